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
constexpr int BIG_BM = 128, BIG_BK = 64, BIG_LD = BIG_BK + 8;   // padded LDS rows (bf16)
}

template <int BN, int WAVES_M>
__global__ __launch_bounds__(256) void conv_big_kernel(ConvArgs a) {
  constexpr int BM = BIG_BM, BK = BIG_BK, LD = BIG_LD;
  constexpr int WAVES_N = 4 / WAVES_M;
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int BVEC = BN * BK / 8;                    // 16-byte vectors of a B chunk
  constexpr int BPT = (BVEC + 255) / 256;              // per thread
  __shared__ __attribute__((aligned(16))) bf16_t As[BM * LD];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[BN * LD];
  __shared__ int ktab[1024];                           // per 8-k vector: tap offset | (dy, dx)

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  const int slot = a.slot0 + (int)blockIdx.y;
  const int64_t Mslot = (int64_t)a.nx * a.P;
  const int64_t m0 = (int64_t)blockIdx.x * BM;
  const int n0 = (int)blockIdx.z * BN;
  const bf16_t* __restrict__ Wt = reinterpret_cast<const bf16_t*>(a.wtab[slot]);
  const int kvec = (a.K + 7) / 8;
  for (int v = tid; v < kvec; v += 256) {
    const int k = v * 8, ci = k % a.C, t = k / a.C;
    const int dy = t / a.kw, dx = t % a.kw;
    ktab[v] = ((dy * a.W + dx) * a.C + ci) | (dy << 24) | (dx << 28);
  }

  // the A row this thread gathers
  const int arow = tid >> 1, ahalf = tid & 1;
  const int64_t m = m0 + arow;
  const bool mvalid = m < Mslot;
  int iy0 = 0, ix0 = 0;
  const bf16_t* inrow = reinterpret_cast<const bf16_t*>(a.in.p);
  if (mvalid) {
    const int xi = (int)(m / a.P), p = (int)(m % a.P);
    int oy, ox;
    if (a.pool) {
      const int q = p >> 2, sub = p & 3;
      oy = 2 * (q / a.Wp) + (sub >> 1);
      ox = 2 * (q % a.Wp) + (sub & 1);
    } else {
      oy = p / a.Wc;
      ox = p % a.Wc;
    }
    iy0 = oy * a.stride - a.pad;
    ix0 = ox * a.stride - a.pad;
    inrow += row_index(a.in.mode, (int64_t)slot * a.nx + xi, a.nx, a.x0) * a.in.row_elems +
             ((int64_t)iy0 * a.W + ix0) * a.C;
  }
  __syncthreads();

  uint4 ra[4], rb[BPT];
  auto load_chunk = [&](int kc) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int v = (kc >> 3) + ahalf * 4 + j;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (mvalid && v < kvec) {
        const int code = ktab[v];
        const int dy = (code >> 24) & 15, dx = (code >> 28) & 15;
        const int iy = iy0 + dy, ix = ix0 + dx;
        if (iy >= 0 && iy < a.H && ix >= 0 && ix < a.W)
          val = *reinterpret_cast<const uint4*>(inrow + (code & 0xFFFFFF));
      }
      ra[j] = val;
    }
#pragma unroll
    for (int j = 0; j < BPT; ++j) {
      const int i = tid + j * 256;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (i < BVEC) {
        const int row = i / (BK / 8), kv = i % (BK / 8);
        const int k = kc + kv * 8;
        if (n0 + row < a.Cout && k < a.K)
          val = *reinterpret_cast<const uint4*>(Wt + (int64_t)(n0 + row) * a.K + k);
      }
      rb[j] = val;
    }
  };
  auto store_chunk = [&]() {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      *reinterpret_cast<uint4*>(&As[arow * LD + (ahalf * 4 + j) * 8]) = ra[j];
#pragma unroll
    for (int j = 0; j < BPT; ++j) {
      const int i = tid + j * 256;
      if (i < BVEC) {
        const int row = i / (BK / 8), kv = i % (BK / 8);
        *reinterpret_cast<uint4*>(&Bs[row * LD + kv * 8]) = rb[j];
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
  for (int j = 0; j < TN; ++j) {
    const int n = n0 + wn * WN + j * 16 + (lane & 15);
    if (n >= a.Cout) continue;
    const float bv = bias[n];
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int64_t mb = m0 + wm * WM + i * 16 + (lane >> 4) * 4;
      if (mb >= Mslot) continue;
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[e] = acc[i][j][e] + bv;
        if (a.relu) v[e] = fmaxf(v[e], 0.f);
      }
      if (a.pool) {
        const float mx = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
        const int xo = (int)(mb / a.P);
        const int q = (int)(mb % a.P) >> 2;
        const int64_t ro = row_index(a.out_mode, (int64_t)slot * a.nx + xo, a.nx, a.x0);
        store_out<bf16_t>(a.out, a.out_f32, ro * a.out_row + (int64_t)q * a.Cout + n, mx);
      } else {
        const int xo = (int)(mb / a.P);
        const int pp = (int)(mb % a.P);
        // the 4 rows of a lane are consecutive pixels of one input (P % 4 == 0)
        const int64_t ro = row_index(a.out_mode, (int64_t)slot * a.nx + xo, a.nx, a.x0);
#pragma unroll
        for (int e = 0; e < 4; ++e)
          store_out<bf16_t>(a.out, a.out_f32, ro * a.out_row + (int64_t)(pp + e) * a.Cout + n, v[e]);
      }
    }
  }
}

int conv_big_bn(int cout) { return cout <= 16 ? 16 : cout <= 32 ? 32 : cout <= 64 ? 64 : 128; }

hipError_t launch_conv_big(const ConvArgs& a, int nslots, hipStream_t s) {
  if (nslots <= 0 || a.nx <= 0) return hipSuccess;
  if (a.C % 8 || a.K > 8 * 1024 || a.P % 4) return hipErrorInvalidValue;
  const int bn = conv_big_bn(a.Cout);
  const int64_t Mslot = (int64_t)a.nx * a.P;
  dim3 grid((unsigned)((Mslot + BIG_BM - 1) / BIG_BM), (unsigned)nslots, (unsigned)((a.Cout + bn - 1) / bn));
  switch (bn) {
    case 16: hipLaunchKernelGGL((conv_big_kernel<16, 4>), grid, dim3(256), 0, s, a); break;
    case 32: hipLaunchKernelGGL((conv_big_kernel<32, 4>), grid, dim3(256), 0, s, a); break;
    case 64: hipLaunchKernelGGL((conv_big_kernel<64, 4>), grid, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((conv_big_kernel<128, 2>), grid, dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

}  // namespace mure
