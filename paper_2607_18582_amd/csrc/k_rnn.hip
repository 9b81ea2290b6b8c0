// Sequence layers of the RNN family (float32 models).
//
// embed_kernel: one thread per (row, step, feature) gathers W[token][d] (the
// library keeps embedding tables token-major, so a token's D values are one
// contiguous row); blocks of one launch row split over the slots.
//
// lstm_kernel: a block owns 64 rows (inputs) of one mutant slot and runs all T
// steps; its waves run independently (each owns 16 rows).  The slot's weights sit in LDS k-major ([D + H + 1][4H]); each wave
// keeps its 16 rows' step input [x_t, h_{t-1}, 1] in LDS and per step computes
// the 4H gate pre-activations as one 16 x 4H GEMM on MFMA
// (v_mfma_f32_16x16x4_f32).  Gate q of unit j is column q*H + j, so with H a
// multiple of 16 one lane holds all four gates of its units in the same
// accumulator position: the cell state stays in registers and the gates never
// leave the lane.
//
// lstm_wide_kernel: for layers whose weights do not fit in LDS.  A block owns
// 64 rows of one slot with H / 16 waves; wave w owns units 16w .. 16w + 15, all
// four gates (64 GEMM columns), and holds its weight columns in registers.
// The step input [x_t, h_{t-1}, 1] lives in LDS as [k / 4][row][4], so the A
// fragments of a k-step are 256 contiguous bytes; two such tiles alternate by
// step: x_{t+1} is fetched into the other tile with direct global-to-LDS
// loads during step t and the gates write h_t there, so one barrier per step
// suffices.
// Both kernels accumulate k in the same order (steps of 4 from k = 0).
#include "dev.hpp"
#include "plan.hpp"

namespace mure {

// VEC features per thread (4: D % 4 == 0, 16-byte loads and stores).
template <int VEC>
__global__ __launch_bounds__(256) void embed_kernel(SeqArgs a, DivU32 dd, DivU32 dt) {
  typedef float vf __attribute__((ext_vector_type(VEC)));
  const int sl = a.slot0 + (int)blockIdx.y;
  const int DV = a.D / VEC;
  const int total = a.nx * a.T * DV;                   // < 2^31 (checked by the launcher)
  const float* __restrict__ X = reinterpret_cast<const float*>(a.in.p);
  const float* __restrict__ Wt = reinterpret_cast<const float*>(a.wtab[sl]);
  for (int i = (int)blockIdx.x * 256 + threadIdx.x; i < total; i += (int)gridDim.x * 256) {
    int rt, dv, xi, t;
    divmodu(dd, (uint32_t)i, rt, dv);                  // rt = xi * T + t
    divmodu(dt, (uint32_t)rt, xi, t);
    const int64_t r = (int64_t)sl * a.nx + xi;
    const float tokf = X[row_index(a.in.mode, r, a.nx, a.x0) * a.in.row_elems + t];
    const int tok = (int)tokf;
    // an id outside the vocabulary (or not an integer) embeds to zeros
    vf v = {};
    if ((float)tok == tokf && tok >= 0 && tok < a.V) v = *reinterpret_cast<const vf*>(Wt + (int64_t)tok * a.D + dv * VEC);
    *reinterpret_cast<vf*>(reinterpret_cast<float*>(a.out) + row_index(a.out_mode, r, a.nx, a.x0) * a.out_row +
                           (int64_t)t * a.D + dv * VEC) = v;
  }
}

// Gate activations from the hardware exponential: sigmoid(z) = 1/(1 + e^-z)
// and tanh(z) = 2 sigmoid(2z) - 1 (a few ulp from the correctly rounded
// values; every launch of a layer uses the same formulas).
__device__ __forceinline__ float sigmoidf_(float z) { return __fdividef(1.f, 1.f + __expf(-z)); }
__device__ __forceinline__ float tanhf_(float z) { return 2.f * sigmoidf_(2.f * z) - 1.f; }

// Zero bytes that the wide kernel's rows past the last input read.
static __device__ __attribute__((aligned(16))) v4f g_lstm_zero[1] = {};
__device__ __forceinline__ const float* lstm_zero() { return reinterpret_cast<const float*>(g_lstm_zero); }

// Block b -> (slot, block of 64 input rows).  Block b runs on XCD b % 8; on
// one XCD consecutive blocks take every slot of one row block in turn, so a
// row block of a shared input (a prefix-cache tensor, read by every slot)
// comes from HBM once and the other slots' reads hit that XCD's L2.  false:
// padding of that order.
__device__ __forceinline__ bool lstm_decode(const SeqArgs& a, int& sl, int& rb) {
  const int b = (int)blockIdx.x, turn = b >> 3;
  rb = (turn / a.nslots) * 8 + (b & 7);
  sl = a.slot0 + turn % a.nslots;
  return rb * 64 < a.nx;
}

template <int HT>                                      // H = 16 * HT units
__global__ __launch_bounds__(256) void lstm_kernel(SeqArgs a) {
  extern __shared__ __attribute__((aligned(16))) float lsm[];
  constexpr int H = 16 * HT, NT = 4 * HT, NS = 4 * H + 16;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int sl, rb;
  if (!lstm_decode(a, sl, rb)) return;
  const int D = a.D, K = D + H + 1;
  const int KP = lstm_kpad(D, H), KA = lstm_ka(D, H);
  float* Ws = lsm;                                     // [KP][NS]
  float* As = lsm + KP * NS;                           // [64][KA]
  const float* __restrict__ Wt = reinterpret_cast<const float*>(a.wtab[sl]);
  // weights: unit j, gate q, k -> Ws[k][q*H + j]
  for (int e = tid; e < KP * 4 * H; e += 256) {
    const int k = e / (4 * H), n = e - k * (4 * H);
    const int q = n / H, j = n - q * H;
    Ws[k * NS + n] = k < K ? Wt[((int64_t)j * 4 + q) * K + k] : 0.f;
  }
  // step tile: x_t (filled per step), h = 0, the bias input 1, zero padding
  for (int e = tid; e < 64 * KA; e += 256) {
    const int k = e % KA;
    As[e] = k == D + H ? 1.f : 0.f;
  }
  __syncthreads();

  const int xi0 = rb * 64 + wave * 16;                 // this wave's 16 rows
  const float* __restrict__ X = reinterpret_cast<const float*>(a.in.p);
  float* __restrict__ Y = reinterpret_cast<float*>(a.out);
  float* A = As + wave * 16 * KA;
  float cst[HT][4];
#pragma unroll
  for (int jj = 0; jj < HT; ++jj)
#pragma unroll
    for (int e = 0; e < 4; ++e) cst[jj][e] = 0.f;
  // row r = slot * nx + xi of the chunk: buffer row r, or cache row x0 + xi
  auto in_row = [&](int xi) {
    return a.in.mode == MODE_BUF ? (int64_t)sl * a.nx + xi : (int64_t)a.x0 + xi;
  };
  auto out_row = [&](int xi) {
    return a.out_mode == MODE_BUF ? (int64_t)sl * a.nx + xi : (int64_t)a.x0 + xi;
  };

  // x_t as 16-byte vectors (D % 4 == 0, at most NXV per lane): the vectors of
  // step t + 1 are loaded during step t, ahead of that step's stores, so
  // their wait does not include the stores; otherwise one element at a time
  constexpr int NXV = 4;
  const int DV = D / 4;
  const bool xvec = D % 4 == 0 && a.in.row_elems % 4 == 0 && 16 * DV <= 64 * NXV;
  int64_t xg[NXV];                                     // element offset of the vector at t = 0, or -1
  int xa[NXV];                                         // its place in A, or -1
  v4f xr[NXV];
#pragma unroll
  for (int u = 0; u < NXV; ++u) {
    const int e4 = lane + 64 * u;
    xg[u] = -1;
    xa[u] = -1;
    if (xvec && e4 < 16 * DV) {
      const int rr = e4 / DV, d4 = e4 - rr * DV;
      xa[u] = rr * KA + d4 * 4;
      if (xi0 + rr < a.nx) xg[u] = in_row(xi0 + rr) * a.in.row_elems + d4 * 4;
    }
  }
  auto load_x = [&](int t) {
#pragma unroll
    for (int u = 0; u < NXV; ++u)
      if (xg[u] >= 0) xr[u] = *reinterpret_cast<const v4f*>(X + xg[u] + (int64_t)t * D);
  };
  if (xvec) load_x(0);
  // h of the previous step, stored to the output during the next step
  float hp[HT][4];
  auto store_h = [&](int t) {
#pragma unroll
    for (int jj = 0; jj < HT; ++jj)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int xi = xi0 + (lane >> 4) * 4 + e;
        if (xi < a.nx)
          Y[out_row(xi) * a.out_row + (int64_t)(a.seq ? t : 0) * H + jj * 16 + (lane & 15)] = hp[jj][e];
      }
  };

  for (int t = 0; t < a.T; ++t) {
    // x_t of the wave's rows (rows past nx read zeros)
    if (xvec) {
#pragma unroll
      for (int u = 0; u < NXV; ++u)
        if (xa[u] >= 0) *reinterpret_cast<v4f*>(A + xa[u]) = xg[u] >= 0 ? xr[u] : v4f{0.f, 0.f, 0.f, 0.f};
      if (t + 1 < a.T) load_x(t + 1);
    } else {
      for (int e = lane; e < 16 * D; e += 64) {
        const int rr = e / D, d = e - rr * D;
        const int xi = xi0 + rr;
        float v = 0.f;
        if (xi < a.nx) v = X[in_row(xi) * a.in.row_elems + (int64_t)t * D + d];
        A[rr * KA + d] = v;
      }
    }
    // a wave reads and writes only its own 16 rows of A, and one wave's LDS
    // operations complete in the order they are issued: no block barrier
    v4f acc[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[j] = v4f{0.f, 0.f, 0.f, 0.f};
    for (int ks = 0; ks < KP; ks += 4) {
      const int k = ks + (lane >> 4);
      const float av = A[(lane & 15) * KA + k];
#pragma unroll
      for (int j = 0; j < NT; ++j)
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, Ws[k * NS + j * 16 + (lane & 15)], acc[j], 0, 0, 0);
    }
    if (a.seq && t > 0) store_h(t - 1);
    // gates: unit u = 16*jj + (lane & 15), rows 4*(lane >> 4) + e of the wave
#pragma unroll
    for (int jj = 0; jj < HT; ++jj) {
      const int u = jj * 16 + (lane & 15);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float ig = sigmoidf_(acc[0 * HT + jj][e]);
        const float fg = sigmoidf_(acc[1 * HT + jj][e]);
        const float gg = tanhf_(acc[2 * HT + jj][e]);
        const float og = sigmoidf_(acc[3 * HT + jj][e]);
        const float c = fmaf(fg, cst[jj][e], ig * gg);
        cst[jj][e] = c;
        const float h = og * tanhf_(c);
        A[((lane >> 4) * 4 + e) * KA + D + u] = h;
        hp[jj][e] = h;
      }
    }
  }
  if (a.T > 0) store_h(a.T - 1);
}


// KS k-steps of 4 (K = D + H + 1 padded with zero weights to 4 KS; the
// launcher rounds the needed steps up to a multiple of 4).
template <int KS>
__global__ __launch_bounds__(256, 1) void lstm_wide_kernel(SeqArgs a) {
  extern __shared__ __attribute__((aligned(16))) float lsm[];
  typedef __attribute__((address_space(3))) void lds_void;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int NW = (int)blockDim.x / 64;                 // = H / 16
  int sl, rb;
  if (!lstm_decode(a, sl, rb)) return;
  const int D = a.D, H = a.H, K = D + H + 1, DS = D / 4;
  // LDS: two step tiles [KS][64][4]: [x_t, h_{t-1}, 1, zeros] of step t in
  // tile t % 2
  const float* __restrict__ Wt = reinterpret_cast<const float*>(a.wtab[sl]);
  const int unit = wave * 16 + (lane & 15);
  // the wave's weight columns: wreg[s][q] = W[unit][gate q][4 s + (lane >> 4)]
  float wreg[KS][4];
#pragma unroll
  for (int s = 0; s < KS; ++s)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int k = 4 * s + (lane >> 4);
      wreg[s][q] = k < K ? Wt[((int64_t)unit * 4 + q) * K + k] : 0.f;
    }
  // both tiles: h = 0, the bias input 1 (k = D + H), zero padding (x_0 is loaded below)
  for (int e = tid; e < 2 * (KS - DS) * 256; e += NW * 64) {
    const int b = e / ((KS - DS) * 256), r = e % ((KS - DS) * 256);
    const int k = D + (r >> 8) * 4 + (r & 3);
    lsm[(b * KS + DS) * 256 + r] = k == D + H ? 1.f : 0.f;
  }
  const int xi0 = rb * 64;
  const float* __restrict__ X = reinterpret_cast<const float*>(a.in.p);
  float* __restrict__ Y = reinterpret_cast<float*>(a.out);
  auto in_row = [&](int xi) {
    return a.in.mode == MODE_BUF ? (int64_t)sl * a.nx + xi : (int64_t)a.x0 + xi;
  };
  auto out_row = [&](int xi) {
    return a.out_mode == MODE_BUF ? (int64_t)sl * a.nx + xi : (int64_t)a.x0 + xi;
  };
  // x_t into tile b: instruction j (channels 4j .. 4j + 3 of the 64 rows),
  // lane = row; rows past nx read the zero page
  const float* xsrc = xi0 + lane < a.nx ? X + in_row(xi0 + lane) * a.in.row_elems : nullptr;
  auto fetch_x = [&](int t, int b) {
    for (int j = wave; j < DS; j += NW)
      __builtin_amdgcn_global_load_lds((const void*)(xsrc ? xsrc + (int64_t)t * D + 4 * j : lstm_zero()),
                                       (lds_void*)(lsm + (b * KS + j) * 256), 16, 0, 0);
  };
  fetch_x(0, 0);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  float cst[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) cst[i][e] = 0.f;
  for (int t = 0; t < a.T; ++t) {
    const int b = t & 1;
    // x_{t+1} and h_t go to the other tile, which no wave reads during step t
    if (t + 1 < a.T) fetch_x(t + 1, b ^ 1);
    // z = [x_t, h_{t-1}, 1] W^T for the wave's 64 columns, k in steps of 4;
    // A fragment: row 16 i + (lane & 15), k = 4 s + (lane >> 4)
    v4f acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[i][q] = v4f{0.f, 0.f, 0.f, 0.f};
    const float* at = lsm + b * KS * 256 + (lane & 15) * 4 + (lane >> 4);
    // the fragments of k-step s + 1 are read before the MFMAs of step s
    float av[2][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) av[0][i] = at[i * 64];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      if (s + 1 < KS) {
#pragma unroll
        for (int i = 0; i < 4; ++i) av[(s + 1) & 1][i] = at[(s + 1) * 256 + i * 64];
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          acc[i][q] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s & 1][i], wreg[s][q], acc[i][q], 0, 0, 0);
    }
    // gates of unit `unit`, rows 16 i + 4 (lane >> 4) + e
    float* hn = lsm + ((b ^ 1) * KS + DS + (unit >> 2)) * 256 + (unit & 3);
    float hv[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float ig = sigmoidf_(acc[i][0][e]);
        const float fg = sigmoidf_(acc[i][1][e]);
        const float gg = tanhf_(acc[i][2][e]);
        const float og = sigmoidf_(acc[i][3][e]);
        const float c = fmaf(fg, cst[i][e], ig * gg);
        cst[i][e] = c;
        const float h = og * tanhf_(c);
        hn[(i * 16 + (lane >> 4) * 4 + e) * 4] = h;
        hv[i][e] = h;
      }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // x_{t+1} has landed
    if (a.seq || t + 1 == a.T) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int xi = xi0 + i * 16 + (lane >> 4) * 4 + e;
          if (xi < a.nx) Y[out_row(xi) * a.out_row + (int64_t)(a.seq ? t : 0) * H + unit] = hv[i][e];
        }
    }
    __syncthreads();                                   // h_t and x_{t+1} in place
  }
}

hipError_t launch_embed(const SeqArgs& a, hipStream_t s) {
  if (a.nslots <= 0 || a.nx <= 0) return hipSuccess;
  const int vec = a.D % 4 == 0 && a.out_row % 4 == 0 ? 4 : 1;
  const int64_t per_slot = (int64_t)a.nx * a.T * (a.D / vec);
  if ((int64_t)a.nx * a.T * a.D >= INT32_MAX || a.nslots > 65535) return hipErrorInvalidValue;
  const int64_t blocks = std::min<int64_t>((per_slot + 255) / 256, 4096);
  const dim3 grid((unsigned)blocks, (unsigned)a.nslots);
  if (vec == 4)
    hipLaunchKernelGGL(embed_kernel<4>, grid, dim3(256), 0, s, a, make_divu32((uint32_t)(a.D / 4)), make_divu32((uint32_t)a.T));
  else
    hipLaunchKernelGGL(embed_kernel<1>, grid, dim3(256), 0, s, a, make_divu32((uint32_t)a.D), make_divu32((uint32_t)a.T));
  return hipGetLastError();
}

hipError_t launch_lstm(const SeqArgs& a, hipStream_t s) {
  if (a.nslots <= 0 || a.nx <= 0) return hipSuccess;
  if (a.H % 16 || a.H < 16 || a.H > 64 || a.nslots > 65535) return hipErrorInvalidValue;
  const int64_t nblk = ((int64_t)(a.nx + 63) / 64 + 7) / 8 * 8 * a.nslots;
  if (nblk >= INT32_MAX) return hipErrorInvalidValue;
  const dim3 grid((unsigned)nblk);
  if (lstm_uses_wide(a.D, a.H)) {
    if (!lstm_wide_fits(a.D, a.H) || a.in.row_elems % 4) return hipErrorInvalidValue;
    const int ks = lstm_wide_ks(a.D, a.H);
    const size_t lds = (size_t)lstm_wide_lds_bytes(a.D, a.H);
    const dim3 block(64 * (a.H / 16));
    switch (ks) {
#define MURE_LSTM_WIDE(n) case n: hipLaunchKernelGGL(lstm_wide_kernel<n>, grid, block, lds, s, a); break;
      MURE_LSTM_WIDE(8) MURE_LSTM_WIDE(12) MURE_LSTM_WIDE(16) MURE_LSTM_WIDE(20) MURE_LSTM_WIDE(24)
      MURE_LSTM_WIDE(28) MURE_LSTM_WIDE(32) MURE_LSTM_WIDE(36) MURE_LSTM_WIDE(40) MURE_LSTM_WIDE(44)
      MURE_LSTM_WIDE(48) MURE_LSTM_WIDE(52)
#undef MURE_LSTM_WIDE
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  const size_t lds = (size_t)lstm_lds_bytes(a.D, a.H);
  if (lds > 64 * 1024) return hipErrorInvalidValue;
  switch (a.H / 16) {
    case 1: hipLaunchKernelGGL(lstm_kernel<1>, grid, dim3(256), lds, s, a); break;
    case 2: hipLaunchKernelGGL(lstm_kernel<2>, grid, dim3(256), lds, s, a); break;
    case 3: hipLaunchKernelGGL(lstm_kernel<3>, grid, dim3(256), lds, s, a); break;
    default: hipLaunchKernelGGL(lstm_kernel<4>, grid, dim3(256), lds, s, a); break;
  }
  return hipGetLastError();
}

}  // namespace mure
