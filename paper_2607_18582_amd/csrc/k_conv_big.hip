// bf16 convolutions with C_in a multiple of 8 as a tiled implicit GEMM on
// MFMA (v_mfma_f32_16x16x32_bf16).
//
// Block tile: 128 GEMM rows (output pixels of (slot, input) rows, pool-window
// major when pooling) x BN output channels, k in chunks of 64.  The im2col
// gather moves 16-byte vectors -- 8 consecutive input channels of one filter
// tap.  The next chunk's global loads are issued before the current chunk's
// MFMAs (register prefetch).
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

// a 16-byte vector in global memory (weight rows are reached through pointer
// tables, which the compiler cannot place in an address space by itself)
typedef __attribute__((address_space(1))) const v4u gv4u;

// LINE (C_in % 64 == 0): a chunk of 64 k is 64 channels of one tap, a whole
// 128-byte line of each row's input pixel.  A thread gathers vector tid % 8
// of rows tid / 8 + (THREADS / 8) r, so a load instruction reads eight whole
// lines instead of 16 bytes from each of 64; the chunk's tap is the same for
// every lane.  Otherwise a thread gathers one row's half chunk of 32 k, in
// groups of G 16-byte vectors of one tap -- G = 4 when C_in % 32 == 0, 2 when
// C_in % 16 == 0, else 1 -- whose tap is the same for the whole wavefront;
// with 16-32 channels consecutive rows' vectors are neighbours in memory.
//
// The 128-row tiles are compiled for three (BN = 128) and five (BN = 64; four
// with LINE, whose four rows per thread need more registers) resident waves
// per SIMD, without spills; their LDS (37 and 28 KB per block) admits that
// many blocks.
template <int BM, int BN, int WAVES_M, int WAVES_N, int G, bool LINE>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N, BM == 128 && BN == 128 ? 3 : BM == 128 && BN == 64 ? (LINE ? 4 : 5) : 1)
void conv_big_kernel(ConvArgs a) {
  constexpr int THREADS = 64 * WAVES_M * WAVES_N;
  constexpr int BK = BIG_BK, LD = BIG_LD;
  constexpr int LPR = LINE ? 8 : 2;                     // threads per A row
  constexpr int ROWS_PER_THREAD = BM * LPR / THREADS;   // A rows gathered by each thread
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int BVEC = BN * BK / 8;                    // 16-byte vectors of a B chunk
  constexpr int BPT = (BVEC + THREADS - 1) / THREADS;  // per thread
  __shared__ __attribute__((aligned(16))) bf16_t smem[(BM + BN) * LD];
  bf16_t* const As = smem;
  bf16_t* const Bs = smem + BM * LD;
  // the epilogue stages each wave's rounded tile here: WM x (WN + 8) per wave
  constexpr bool STAGE_FITS = BM * (BN + 8 * WAVES_N) <= (BM + BN) * LD;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  // Tile order.  LINE: XCD-aware -- block b runs on XCD b % 8, and each XCD
  // takes a contiguous run of (slot, row tile, column block) tiles, column
  // blocks innermost, so the tiles running together on it are neighbouring
  // row tiles of one slot and share their input rows in its L2 (resnet18w's
  // strided convolutions and projections: 432 -> 408 ms per step).  Narrower
  // inputs keep the 3-D grid (row tiles, slots, column blocks): for their
  // small tiles the decode made resnet20's 16-channel layers 3.5 % slower.
  int bx, by, bz;
  if constexpr (LINE) {
    const int b = (int)blockIdx.x, turns = (int)((gridDim.x + 7) / 8);
    const int idx = (b & 7) * turns + (b >> 3);
    if (idx >= a.big_tiles) return;                    // padding of the order (whole block)
    bz = idx % a.big_gz;
    const int rest = idx / a.big_gz;
    bx = rest % a.big_gx;
    by = rest / a.big_gx;
  } else {
    bx = (int)blockIdx.x;
    by = (int)blockIdx.y;
    bz = (int)blockIdx.z;
  }
  const int slot = a.slot0 + by;
  const int Mslot = a.nx * a.P;                        // < 2^31 (checked by the launcher)
  const int m0 = bx * BM;
  const int n0 = bz * BN;
  const bf16_t* __restrict__ Wt = reinterpret_cast<const bf16_t*>(a.wtab[slot]);
  const int ncol = a.cols ? a.ncols : a.Cout;
  const bf16_t* const zp = reinterpret_cast<const bf16_t*>(g_zero_page);

  // the A rows this thread gathers: rows arow + RSTEP r; LINE: vector av of
  // each, else k half av (a wave covers 64 consecutive rows of one half, so
  // its 16-byte LDS stores hit distinct banks)
  constexpr int RSTEP = THREADS / LPR;
  const int arow = LINE ? tid / 8 : tid % RSTEP;
  const int av = LINE ? tid % 8 : __builtin_amdgcn_readfirstlane(tid / RSTEP);
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

  constexpr int VPT = LINE ? 1 : 4;                    // 16-byte vectors per row per thread
  v4u ra[ROWS_PER_THREAD][VPT], rb[BPT];
  auto load_chunk = [&](int kc) {
    if constexpr (LINE) {
      // the chunk's tap t (wave-uniform) and this thread's channels ci
      int t, c0, dy, dx;
      divmodu(a.dC, (uint32_t)kc, t, c0);
      divmodu(a.dKW, (uint32_t)t, dy, dx);
      const int off = (dy * a.W + dx) * a.C + c0 + av * 8;
#pragma unroll
      for (int r = 0; r < ROWS_PER_THREAD; ++r) {
        const int iy = iy0[r] + dy, ix = ix0[r] + dx;
        const bool ok = (unsigned)iy < (unsigned)a.H && (unsigned)ix < (unsigned)a.W;
        ra[r][0] = *reinterpret_cast<const v4u*>(ok ? inrow[r] + off : zp);
      }
    } else {
#pragma unroll
      for (int jg = 0; jg < 4; jg += G) {
        // k of this group (wave-uniform): tap t, first channel ci
        const int k = kc + av * 32 + jg * 8;
        int t, ci, dy, dx;
        divmodu(a.dC, (uint32_t)k, t, ci);
        divmodu(a.dKW, (uint32_t)t, dy, dx);
        const int off = (dy * a.W + dx) * a.C + ci;
        if (k >= a.K) dy = -(1 << 20);               // past the end: every row reads zeros
#pragma unroll
        for (int r = 0; r < ROWS_PER_THREAD; ++r) {
          const int iy = iy0[r] + dy, ix = ix0[r] + dx;
          const bool ok = (unsigned)iy < (unsigned)a.H && (unsigned)ix < (unsigned)a.W;
          const v4u* src = reinterpret_cast<const v4u*>(ok ? inrow[r] + off : zp);
#pragma unroll
          for (int g = 0; g < G; ++g) ra[r][jg + g] = src[g];
        }
      }
    }
#pragma unroll
    for (int j = 0; j < BPT; ++j) {
      // past the last column or the row's end: the zero page (a select, not a branch)
      const int i = tid + j * THREADS;
      const bf16_t* src = brow[j] && kc + (i % (BK / 8)) * 8 < a.K ? brow[j] + kc : zp;
      rb[j] = *(const gv4u*)src;
    }
  };
  auto store_chunk = [&]() {
#pragma unroll
    for (int r = 0; r < ROWS_PER_THREAD; ++r)
#pragma unroll
      for (int j = 0; j < VPT; ++j)
        *reinterpret_cast<v4u*>(&As[(arow + RSTEP * r) * LD + (LINE ? av : av * 4 + j) * 8]) = ra[r][j];
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

  auto mma_step = [&](int ks) {
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
  };

  load_chunk(0);
  for (int kc = 0; kc < a.K; kc += BK) {
    store_chunk();
    __syncthreads();
    if (kc + BK < a.K) load_chunk(kc + BK);             // next chunk in flight
    // the tail's k past K holds zeros on both operands (adding +0 products);
    // one straight-line body keeps the accumulators in AGPRs across the loop
    mma_step(0);
    mma_step(1);
    __syncthreads();
  }

  const float* __restrict__ bias = a.btab[slot];
  if constexpr (STAGE_FITS) {
    if (!a.cols && a.Cout % 8 == 0 && !a.out_f32 && (a.add_mode == 0 || (a.add_mode == 1 && !a.add_out_f32))) {
      // Round the wave's tile into LDS (bias, ReLU, pool applied), then store
      // whole 16-byte channel vectors: rows of the output are [pixel][C_out].
      constexpr int OLD = WN + 8;
      bf16_t* Os = smem + wave * WM * OLD;
      const int RW = a.pool ? WM / 4 : WM;               // staged rows
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int nl = j * 16 + (lane & 15);
        const int n = n0 + wn * WN + nl;
        const float bv = n < a.Cout ? bias[n] : 0.f;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[e] = acc[i][j][e] + bv;
            v[e] = act(v[e], a.relu);
          }
          if (a.pool) {
            Os[(i * 4 + (lane >> 4)) * OLD + nl] = f2bf(fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3])));
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) Os[(i * 16 + (lane >> 4) * 4 + e) * OLD + nl] = f2bf(v[e]);
          }
        }
      }
      __syncthreads();                                   // the staged tiles are complete
      const int Mout = a.pool ? Mslot / 4 : Mslot;
      const int g0 = (m0 + wm * WM) / (a.pool ? 4 : 1);
      const DivU32 dpo = a.pool ? a.dPq : a.dP;
      for (int idx = lane; idx < RW * (WN / 8); idx += 64) {
        const int row = idx / (WN / 8), vc = idx % (WN / 8);
        const int g = g0 + row;
        const int n = n0 + wn * WN + vc * 8;
        if (g >= Mout || n >= a.Cout) continue;
        int xo, q;
        divmodu(dpo, (uint32_t)g, xo, q);
        const int64_t ro = row_index(a.out_mode, (int64_t)slot * a.nx + xo, a.nx, a.x0);
        v4u val = *reinterpret_cast<const v4u*>(&Os[row * OLD + vc * 8]);
        if (a.add_mode == 1) {
          // conv_b's rounded output + the identity shortcut, in float32, then ReLU
          const v4u sk = *reinterpret_cast<const v4u*>(
              reinterpret_cast<const bf16_t*>(a.skip.p) +
              row_index(a.skip.mode, (int64_t)slot * a.nx + xo, a.nx, a.x0) * a.skip.row_elems +
              (int64_t)q * a.Cout + n);
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            uint32_t o = 0;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              float t = bf2f((bf16_t)(val[w] >> (16 * h))) + bf2f((bf16_t)(sk[w] >> (16 * h)));
              t = act(t, a.add_relu);
              o |= (uint32_t)f2bf(t) << (16 * h);
            }
            val[w] = o;
          }
        }
        *reinterpret_cast<v4u*>(reinterpret_cast<bf16_t*>(a.out) + ro * a.out_row + (int64_t)q * a.Cout + n) = val;
      }
      return;
    }
  }
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
        v[e] = act(v[e], a.relu);
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
          t = act(t, a.add_relu);
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

template <int G, bool LINE>
static hipError_t launch_big(const ConvArgs& a, dim3 grid, int bm, int bn, hipStream_t s) {
  if (bm == 128) {
    switch (bn) {
      case 16: hipLaunchKernelGGL((conv_big_kernel<128, 16, 4, 1, G, LINE>), grid, dim3(256), 0, s, a); break;
      case 32: hipLaunchKernelGGL((conv_big_kernel<128, 32, 4, 1, G, LINE>), grid, dim3(256), 0, s, a); break;
      case 64: hipLaunchKernelGGL((conv_big_kernel<128, 64, 4, 1, G, LINE>), grid, dim3(256), 0, s, a); break;
      default: hipLaunchKernelGGL((conv_big_kernel<128, 128, 2, 2, G, LINE>), grid, dim3(256), 0, s, a); break;
    }
  } else {
    switch (bn) {
      case 16: hipLaunchKernelGGL((conv_big_kernel<256, 16, 8, 1, G, LINE>), grid, dim3(512), 0, s, a); break;
      case 32: hipLaunchKernelGGL((conv_big_kernel<256, 32, 8, 1, G, LINE>), grid, dim3(512), 0, s, a); break;
      case 64: hipLaunchKernelGGL((conv_big_kernel<256, 64, 4, 2, G, LINE>), grid, dim3(512), 0, s, a); break;
      default: hipLaunchKernelGGL((conv_big_kernel<256, 128, 4, 2, G, LINE>), grid, dim3(512), 0, s, a); break;
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
  const int64_t gx = (Mslot + bm - 1) / bm, gz = (ncol + bn - 1) / bn;
  const int64_t tiles = gx * nslots * gz;
  if (tiles >= (1 << 30)) return hipErrorInvalidValue;
  a.big_gx = (int)gx;
  a.big_gz = (int)gz;
  a.big_tiles = (int)tiles;
  const dim3 grid = a.C % 64 == 0 ? dim3((unsigned)((tiles + 7) / 8 * 8))
                                  : dim3((unsigned)gx, (unsigned)nslots, (unsigned)gz);
  a.dPq = make_divu32((uint32_t)std::max(1, a.P / 4));
  a.dC = make_divu32((uint32_t)a.C);
  a.dKW = make_divu32((uint32_t)a.kw);
  if (a.C % 64 == 0) return launch_big<4, true>(a, grid, bm, bn, s);
  if (a.C % 32 == 0) return launch_big<4, false>(a, grid, bm, bn, s);
  if (a.C % 16 == 0) return launch_big<2, false>(a, grid, bm, bn, s);
  return launch_big<1, false>(a, grid, bm, bn, s);
}

}  // namespace mure
