// bf16 convolutions with C_in a multiple of 8 as a tiled implicit GEMM on
// MFMA (v_mfma_f32_16x16x32_bf16).
//
// Block tile: 128 GEMM rows (output pixels of (slot, input) rows, pool-window
// major when pooling) x BN output channels, k in chunks of 64.  The im2col
// gather moves 16-byte vectors -- 8 consecutive input channels of one filter
// tap -- guided by a per-block table of the taps; the next chunk's global
// loads are issued before the current chunk's MFMAs (register prefetch).
// Reduction order: k = (dy, dx, c_in), c_in fastest, in increasing steps of
// 32 with zero padding, for every launch of a node.
#include "dev.hpp"
#include "plan.hpp"

namespace mure {

namespace {
constexpr int BIG_BK = 64, BIG_LD = BIG_BK + 8;   // padded LDS rows (bf16)
}

// Zero bytes that out-of-image taps and rows past the end read instead of the
// input, so every gather is an unconditional 16-byte load.
static __device__ __attribute__((aligned(16))) v4u g_zero_page[16] = {};

// TAP64: C_in % 64 == 0, so every 64-wide k chunk lies inside one filter tap
// and each thread's 4 vectors are 64 contiguous bytes of one input pixel (one
// bounds check, one address per chunk).
template <int BM, int BN, int WAVES_M, int WAVES_N, bool TAP64>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N)
void conv_big_kernel(ConvArgs a) {
  constexpr int THREADS = 64 * WAVES_M * WAVES_N;
  constexpr int BK = BIG_BK, LD = BIG_LD;
  constexpr int ROWS_PER_THREAD = BM * 2 / THREADS;   // A rows gathered by each thread (2 per row)
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int BVEC = BN * BK / 8;                    // 16-byte vectors of a B chunk
  constexpr int BPT = (BVEC + THREADS - 1) / THREADS;  // per thread
  __shared__ __attribute__((aligned(16))) bf16_t As[BM * LD];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[BN * LD];
  __shared__ int ktab[1024];                           // per 8-k vector: tap offset | (dy, dx)

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  const int slot = a.slot0 + (int)blockIdx.y;
  const int Mslot = a.nx * a.P;                        // < 2^31 (checked by the launcher)
  const int m0 = (int)blockIdx.x * BM;
  const int n0 = (int)blockIdx.z * BN;
  const bf16_t* __restrict__ Wt = reinterpret_cast<const bf16_t*>(a.wtab[slot]);
  const int ncol = a.cols ? a.ncols : a.Cout;
  const bf16_t* const zp = reinterpret_cast<const bf16_t*>(g_zero_page);
  const int kvec = (a.K + 7) / 8;
  if constexpr (!TAP64) {
    for (int v = tid; v < kvec; v += THREADS) {
      const int k = v * 8, ci = k % a.C, t = k / a.C;
      const int dy = t / a.kw, dx = t % a.kw;
      ktab[v] = ((dy * a.W + dx) * a.C + ci) | (dy << 24) | (dx << 28);
    }
  }

  // the A rows this thread gathers: rows arow + RSTEP*r, k half ahalf (a wave
  // covers 64 consecutive rows of one half, so its 16-byte LDS stores hit
  // distinct banks)
  constexpr int RSTEP = THREADS / 2;
  const int arow = tid % RSTEP, ahalf = tid / RSTEP;
  bool mvalid[ROWS_PER_THREAD];
  int iy0[ROWS_PER_THREAD], ix0[ROWS_PER_THREAD];
  const bf16_t* inrow[ROWS_PER_THREAD];
#pragma unroll
  for (int r = 0; r < ROWS_PER_THREAD; ++r) {
    const int m = m0 + arow + RSTEP * r;
    mvalid[r] = m < Mslot;
    iy0[r] = ix0[r] = -(1 << 20);                    // rows past the end: every tap out of the image
    inrow[r] = zp;
    if (mvalid[r]) {
      int xi, p, oy, ox;
      divmodu(a.dP, (uint32_t)m, xi, p);
      if (a.pool) {
        int qy, qx;
        divmodu(a.dWp, (uint32_t)(p >> 2), qy, qx);
        oy = 2 * qy + ((p >> 1) & 1);
        ox = 2 * qx + (p & 1);
      } else {
        divmodu(a.dWc, (uint32_t)p, oy, ox);
      }
      iy0[r] = oy * a.stride - a.pad;
      ix0[r] = ox * a.stride - a.pad;
      inrow[r] = reinterpret_cast<const bf16_t*>(a.in.p) +
                 row_index(a.in.mode, (int64_t)slot * a.nx + xi, a.nx, a.x0) * a.in.row_elems +
                 ((int64_t)iy0[r] * a.W + ix0[r]) * a.C;
    }
  }
  // the weight rows this thread loads (a gathered delta takes each column's
  // row from its own mutant's weights); nullptr past the last column
  const bf16_t* brow[BPT];
#pragma unroll
  for (int j = 0; j < BPT; ++j) {
    const int i = tid + j * THREADS;
    const int n = n0 + i / (BK / 8);
    brow[j] = nullptr;
    if (i < BVEC && n < ncol) {
      if (a.cols) {
        const DeltaCol cd = a.cols[n];
        brow[j] = reinterpret_cast<const bf16_t*>(a.wtab[a.slot0 + cd.slot - a.col_slot0]) + (int64_t)cd.c * a.K;
      } else {
        brow[j] = Wt + (int64_t)n * a.K;
      }
      brow[j] += (i % (BK / 8)) * 8;
    }
  }
  __syncthreads();

  v4u ra[ROWS_PER_THREAD][4], rb[BPT];
  auto load_chunk = [&](int kc) {
    if constexpr (TAP64) {
      // chunk kc: tap t = kc / C (uniform), channels ci0 .. ci0 + 63
      const int t = kc / a.C, ci0 = kc - t * a.C;
      const int dy = t / a.kw, dx = t - dy * a.kw;
      const int off = (dy * a.W + dx) * a.C + ci0 + ahalf * 32;
#pragma unroll
      for (int r = 0; r < ROWS_PER_THREAD; ++r) {
        const int iy = iy0[r] + dy, ix = ix0[r] + dx;
        const bool ok = (unsigned)iy < (unsigned)a.H && (unsigned)ix < (unsigned)a.W;
        const v4u* src = reinterpret_cast<const v4u*>(ok ? inrow[r] + off : zp);
#pragma unroll
        for (int j = 0; j < 4; ++j) ra[r][j] = src[j];
      }
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int v = (kc >> 3) + ahalf * 4 + j;
        int code = 0, dy = -(1 << 20), dx = 0;       // k past the end: out of the image
        if (v < kvec) {
          code = ktab[v];
          dy = (code >> 24) & 15;
          dx = (code >> 28) & 15;
        }
#pragma unroll
        for (int r = 0; r < ROWS_PER_THREAD; ++r) {
          const int iy = iy0[r] + dy, ix = ix0[r] + dx;
          const bool ok = (unsigned)iy < (unsigned)a.H && (unsigned)ix < (unsigned)a.W;
          ra[r][j] = *reinterpret_cast<const v4u*>(ok ? inrow[r] + (code & 0xFFFFFF) : zp);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < BPT; ++j) {
      const int i = tid + j * THREADS;
      v4u val = v4u{0u, 0u, 0u, 0u};
      if (brow[j] && kc + (i % (BK / 8)) * 8 < a.K) val = *reinterpret_cast<const v4u*>(brow[j] + kc);
      rb[j] = val;
    }
  };
  auto store_chunk = [&]() {
#pragma unroll
    for (int r = 0; r < ROWS_PER_THREAD; ++r)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        *reinterpret_cast<v4u*>(&As[(arow + RSTEP * r) * LD + (ahalf * 4 + j) * 8]) = ra[r][j];
#pragma unroll
    for (int j = 0; j < BPT; ++j) {
      const int i = tid + j * THREADS;
      if (i < BVEC) {
        const int row = i / (BK / 8), kv = i % (BK / 8);
        *reinterpret_cast<v4u*>(&Bs[row * LD + kv * 8]) = rb[j];
      }
    }
  };

  v4f acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  load_chunk(0);
  for (int kc = 0; kc < a.K; kc += BK) {
    store_chunk();
    __syncthreads();
    if (kc + BK < a.K) load_chunk(kc + BK);             // next chunk in flight
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      v8bf av[TM], bv[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        av[i] = *reinterpret_cast<const v8bf*>(&As[(wm * WM + i * 16 + (lane & 15)) * LD + ks * 32 + (lane >> 4) * 8]);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bv[j] = *reinterpret_cast<const v8bf*>(&Bs[(wn * WN + j * 16 + (lane & 15)) * LD + ks * 32 + (lane >> 4) * 8]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }

  const float* __restrict__ bias = a.btab[slot];
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int mb = m0 + wm * WM + i * 16 + (lane >> 4) * 4;
    if (mb >= Mslot) continue;
    // the 4 rows of a lane are one pool window, or 4 consecutive pixels of one
    // input (P % 4 == 0)
    int xo, pb;
    divmodu(a.dP, (uint32_t)mb, xo, pb);
    const bf16_t* sp = nullptr;
    if (a.add_mode)
      sp = reinterpret_cast<const bf16_t*>(a.skip.p) +
           row_index(a.skip.mode, (int64_t)slot * a.nx + xo, a.nx, a.x0) * a.skip.row_elems;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int nc = n0 + wn * WN + j * 16 + (lane & 15);
      if (nc >= ncol) continue;
      // output slot, channel and channel stride of this column
      int os = slot, n = nc, ostride = a.Cout;
      float bv;
      if (a.cols) {
        const DeltaCol cd = a.cols[nc];
        os = a.slot0 + cd.slot - a.col_slot0;
        bv = a.btab[os][cd.c];
        n = a.delta_T > 0 ? cd.t : cd.c;
        if (a.delta_T > 0) ostride = a.delta_T;
      } else {
        bv = bias[nc];
      }
      const int64_t ro = row_index(a.out_mode, (int64_t)os * a.nx + xo, a.nx, a.x0);
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[e] = acc[i][j][e] + bv;
        if (a.relu) v[e] = fmaxf(v[e], 0.f);
      }
      if (a.pool) {
        const float mx = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
        store_out<bf16_t>(a.out, a.out_f32, ro * a.out_row + (int64_t)(pb >> 2) * ostride + n, mx);
      } else if (a.add_mode) {
        // conv_b's output (rounded) + the shortcut, in float32, then ReLU
        const int cs = a.add_mode == 1 ? n : n - (a.Cout - a.Cs) / 2;
        int y = 0, x = 0;
        if (a.add_mode == 2) divmodu(a.dWc, (uint32_t)pb, y, x);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float sv = 0.f;
          if (a.add_mode == 1) {
            sv = bf2f(sp[(int64_t)(pb + e) * a.Cout + n]);
          } else if (cs >= 0 && cs < a.Cs) {
            sv = bf2f(sp[((int64_t)(2 * y) * a.Ws + 2 * x) * a.Cs + cs]);
          }
          if (a.add_mode == 2 && ++x == a.Wc) { x = 0; ++y; }
          float t = bf2f(f2bf(v[e])) + sv;
          if (a.add_relu) t = fmaxf(t, 0.f);
          store_out<bf16_t>(a.out, a.add_out_f32, ro * a.out_row + (int64_t)(pb + e) * a.Cout + n, t);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          store_out<bf16_t>(a.out, a.out_f32, ro * a.out_row + (int64_t)(pb + e) * ostride + n, v[e]);
      }
    }
  }
}

int conv_big_bn(int cout) { return cout <= 16 ? 16 : cout <= 32 ? 32 : cout <= 64 ? 64 : 128; }

template <bool TAP64>
static hipError_t launch_big(const ConvArgs& a, dim3 grid, int bm, int bn, hipStream_t s) {
  if (bm == 128) {
    switch (bn) {
      case 16: hipLaunchKernelGGL((conv_big_kernel<128, 16, 4, 1, TAP64>), grid, dim3(256), 0, s, a); break;
      case 32: hipLaunchKernelGGL((conv_big_kernel<128, 32, 4, 1, TAP64>), grid, dim3(256), 0, s, a); break;
      case 64: hipLaunchKernelGGL((conv_big_kernel<128, 64, 4, 1, TAP64>), grid, dim3(256), 0, s, a); break;
      default: hipLaunchKernelGGL((conv_big_kernel<128, 128, 2, 2, TAP64>), grid, dim3(256), 0, s, a); break;
    }
  } else {
    switch (bn) {
      case 16: hipLaunchKernelGGL((conv_big_kernel<256, 16, 8, 1, TAP64>), grid, dim3(512), 0, s, a); break;
      case 32: hipLaunchKernelGGL((conv_big_kernel<256, 32, 8, 1, TAP64>), grid, dim3(512), 0, s, a); break;
      case 64: hipLaunchKernelGGL((conv_big_kernel<256, 64, 4, 2, TAP64>), grid, dim3(512), 0, s, a); break;
      default: hipLaunchKernelGGL((conv_big_kernel<256, 128, 4, 2, TAP64>), grid, dim3(512), 0, s, a); break;
    }
  }
  return hipGetLastError();
}

hipError_t launch_conv_big(const ConvArgs& a0, int nslots, hipStream_t s) {
  if (nslots <= 0 || a0.nx <= 0) return hipSuccess;
  if (a0.C % 8 || a0.K > 8 * 1024 || a0.P % 4 || (int64_t)a0.nx * a0.P + 256 >= INT32_MAX)
    return hipErrorInvalidValue;
  if (a0.cols && (a0.in.mode != MODE_CACHE || a0.add_mode || a0.ncols <= 0)) return hipErrorInvalidValue;
  if (a0.cols) nslots = 1;
  ConvArgs a = a0;
  a.dP = make_divu32((uint32_t)a.P);
  a.dWp = make_divu32((uint32_t)std::max(1, a.Wp));
  a.dWc = make_divu32((uint32_t)std::max(1, a.Wc));
  const int bn = conv_big_bn(a.cols ? a.ncols : a.Cout);
  // tile: 0 automatic, 1 = 128 rows x BN (4 waves), 2 = 256 rows x BN (8 waves of 64 x 32..64)
  const int bm = a.tile == 2 ? 256 : 128;
  const int64_t Mslot = (int64_t)a.nx * a.P;
  const int ncol = a.cols ? a.ncols : a.Cout;
  dim3 grid((unsigned)((Mslot + bm - 1) / bm), (unsigned)nslots, (unsigned)((ncol + bn - 1) / bn));
  if (a.C % 64 == 0) return launch_big<true>(a, grid, bm, bn, s);
  return launch_big<false>(a, grid, bm, bn, s);
}

}  // namespace mure
