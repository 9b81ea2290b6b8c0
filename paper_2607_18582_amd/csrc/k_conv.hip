// The general CONV2D kernel (any shape; here the bf16 stems with C_in = 3):
// an implicit GEMM on MFMA with a scalar im2col gather.
//
// GEMM view of one node over a chunk: rows m = (slot, input, output pixel),
// columns n = output channel, reduction k = (dy, dx, c_in) in the weight
// layout [C_out][kh][kw][C_in] (c_in fastest).  The reduction is accumulated
// in float32 by v_mfma_f32_16x16x4_f32 (fp32 models, 4 k per step) or
// v_mfma_f32_16x16x32_bf16 (bf16 models, 32 k per step) in increasing k,
// zero-padded to a whole step -- every kernel that computes a node uses the
// same steps, so a node's value never depends on which kernel or batch
// produced it.  Epilogue in float32: + bias, ReLU, 2x2 max-pool, then the
// node-output rounding (bf16 round-to-nearest-even, or float32).
//
// With pooling, the rows of one input are ordered pool-window-major
// (window q = py*Wp + px, then its 4 pixels), so the 4 accumulators a lane
// holds for one output column are one pooling window.
#include "dev.hpp"

namespace mure {

template <typename T> struct Mfma;
template <> struct Mfma<float> { static constexpr int BK = 16, PAD = 1; };
template <> struct Mfma<bf16_t> { static constexpr int BK = 32, PAD = 8; };

template <typename T, int BM, int BN>
__global__ __launch_bounds__(256) void conv_mfma_kernel(ConvArgs a) {
  static_assert(BM == 64 && BN == 64, "tile");
  constexpr int BK = Mfma<T>::BK;
  constexpr int LDA = BK + Mfma<T>::PAD;
  constexpr int EPT = BK / 4;
  __shared__ __attribute__((aligned(16))) T As[BM * LDA];
  __shared__ __attribute__((aligned(16))) T Bs[BN * LDA];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int slot = a.slot0 + (int)blockIdx.y;
  const int64_t Mslot = (int64_t)a.nx * a.P;
  const int64_t m_tile0 = (int64_t)blockIdx.x * BM;
  const int n_tile0 = (int)blockIdx.z * BN;
  const T* __restrict__ Wt = reinterpret_cast<const T*>(a.wtab[slot]);
  const int ncol = a.cols ? a.ncols : a.Cout;

  // the A row this thread gathers (fixed for the block)
  const int m_local = tid & (BM - 1);
  const int kq = tid >> 6;
  const int64_t m = m_tile0 + m_local;
  const bool mvalid = m < Mslot;
  int xi = 0, p = 0;
  if (mvalid) { xi = (int)(m / a.P); p = (int)(m % a.P); }
  int oy, ox;
  if (a.pool) {
    const int q = p >> 2, sub = p & 3;
    oy = 2 * (q / a.Wp) + (sub >> 1);
    ox = 2 * (q % a.Wp) + (sub & 1);
  } else {
    oy = p / a.Wc;
    ox = p % a.Wc;
  }
  const int iy0 = oy * a.stride - a.pad, ix0 = ox * a.stride - a.pad;
  const int64_t r = (int64_t)slot * a.nx + xi;
  const T* __restrict__ inrow =
      reinterpret_cast<const T*>(a.in.p) + row_index(a.in.mode, r, a.nx, a.x0) * a.in.row_elems;
  // the B row (output channel) this thread loads
  const int n_ld = n_tile0 + (tid & 63);
  const bool nvalid = n_ld < ncol;
  const T* __restrict__ wrow = Wt;
  if (nvalid) {
    if (a.cols) {   // a gathered delta column: its own mutant's weight row
      const DeltaCol cd = a.cols[n_ld];
      wrow = reinterpret_cast<const T*>(a.wtab[a.slot0 + cd.slot - a.col_slot0]) + (int64_t)cd.c * a.K;
    } else {
      wrow = Wt + (int64_t)n_ld * a.K;
    }
  }

  v4f acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  for (int kc = 0; kc < a.K; kc += BK) {
    {  // A: im2col gather of EPT consecutive k for row m
      int k = kc + kq * EPT;
      int ci = k % a.C, t2 = k / a.C;
      int dx = t2 % a.kw, dy = t2 / a.kw;
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        T v = T(0);
        if (mvalid && k < a.K) {
          const int iy = iy0 + dy, ix = ix0 + dx;
          if (iy >= 0 && iy < a.H && ix >= 0 && ix < a.W) v = inrow[((int64_t)iy * a.W + ix) * a.C + ci];
        }
        As[m_local * LDA + kq * EPT + e] = v;
        ++k;
        if (++ci == a.C) { ci = 0; if (++dx == a.kw) { dx = 0; ++dy; } }
      }
    }
    {  // B: EPT consecutive k of output channel n_ld
      const int k0 = kc + kq * EPT;
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        const int k = k0 + e;
        Bs[(tid & 63) * LDA + kq * EPT + e] = (nvalid && k < a.K) ? wrow[k] : T(0);
      }
    }
    __syncthreads();
    if constexpr (sizeof(T) == 4) {
#pragma unroll
      for (int ks = 0; ks < BK / 4; ++ks) {
        float av[2], bv[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          av[t] = As[(wm * 32 + t * 16 + (lane & 15)) * LDA + ks * 4 + (lane >> 4)];
          bv[t] = Bs[(wn * 32 + t * 16 + (lane & 15)) * LDA + ks * 4 + (lane >> 4)];
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], bv[j], acc[i][j], 0, 0, 0);
      }
    } else {
      v8bf av[2], bv[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        av[t] = *reinterpret_cast<const v8bf*>(&As[(wm * 32 + t * 16 + (lane & 15)) * LDA + (lane >> 4) * 8]);
        bv[t] = *reinterpret_cast<const v8bf*>(&Bs[(wn * 32 + t * 16 + (lane & 15)) * LDA + (lane >> 4) * 8]);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }

  // epilogue: lane holds rows mb..mb+3 of column n
  const float* __restrict__ bias = a.btab[slot];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int nc = n_tile0 + wn * 32 + j * 16 + (lane & 15);
      const int64_t mb = m_tile0 + wm * 32 + i * 16 + (lane >> 4) * 4;
      if (nc >= ncol || mb >= Mslot) continue;
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
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[e] = acc[i][j][e] + bv;
        v[e] = act(v[e], a.relu);
      }
      if (a.pool) {
        const float mx = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
        const int xo = (int)(mb / a.P);
        const int q = (int)(mb % a.P) >> 2;
        const int64_t ro = row_index(a.out_mode, (int64_t)os * a.nx + xo, a.nx, a.x0);
        store_out<T>(a.out, a.out_f32, ro * a.out_row + (int64_t)q * ostride + n, mx);
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int64_t mm = mb + e;
          if (mm >= Mslot) break;
          const int xo = (int)(mm / a.P);
          const int pp = (int)(mm % a.P);
          const int64_t ro = row_index(a.out_mode, (int64_t)os * a.nx + xo, a.nx, a.x0);
          store_out<T>(a.out, a.out_f32, ro * a.out_row + (int64_t)pp * ostride + n, v[e]);
        }
      }
    }
  }
}

hipError_t launch_conv(const ConvArgs& a, int nslots, int dtype, hipStream_t s) {
  if (nslots <= 0 || a.nx <= 0) return hipSuccess;
  if (a.cols && (a.in.mode != MODE_CACHE || a.add_mode || a.ncols <= 0)) return hipErrorInvalidValue;
  if (a.cols) nslots = 1;
  const int64_t Mslot = (int64_t)a.nx * a.P;
  const int ncol = a.cols ? a.ncols : a.Cout;
  dim3 grid((unsigned)((Mslot + 63) / 64), (unsigned)nslots, (unsigned)((ncol + 63) / 64));
  if (dtype == 0)
    hipLaunchKernelGGL((conv_mfma_kernel<float, 64, 64>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((conv_mfma_kernel<bf16_t, 64, 64>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace mure
