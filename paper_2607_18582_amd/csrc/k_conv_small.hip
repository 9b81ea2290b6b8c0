// Convolutions with small images or few output channels.
//
// conv_lds_kernel (fp32): the zero-padded input images a block needs and the
// weight matrix of its output channels live in LDS, so the k loop runs without
// barriers; A operands are read straight from the image through a per-k
// offset table (k = (dy, dx, c_in), c_in fastest).  With C_in odd an MFMA
// takes 4 consecutive k; with C_in even (PAIR) a step of 8 k gives each lane
// group the pair (2g, 2g + 1), adjacent in the image and in the pair-
// interleaved weight tile, so one 8-byte read feeds the two MFMAs of the
// step (even k, then odd k) and the address arithmetic halves.  The order is
// a function of the node's shape, as for every family.  A block keeps its
// weights and walks several 256-row pieces of its slot.  Its input may be "virtual": the first
// mutated node's output seen through the mutant's channel map and compact
// delta rows, so that output is never materialised per mutant.
//
// conv_valu_kernel: C_out below one MFMA tile.  A block stages a few input
// images and the weights in LDS; each thread owns one stored output position
// and accumulates every (pool-window pixel, channel) output as a fused
// multiply-add chain over k in increasing order.  A list of channels per slot
// restricts the work to the channels a fuzz or inverse record changed (the
// delta at the first mutated layer); each output's chain is the same whichever
// channels are computed, so the delta is bit-identical to the full layer.
#include "dev.hpp"
#include "plan.hpp"

namespace mure {

// Waves per SIMD the register budget must allow: the LDS tile of a 16-column
// block leaves room for five or six resident blocks per CU.
template <int BN, bool PAIR>
__global__ __launch_bounds__(256, BN == 16 ? (PAIR ? 6 : 5) : BN == 32 ? 3 : 2) void conv_lds_kernel(ConvArgs a, int nimg_cap, int kpad, int iters) {
  extern __shared__ __attribute__((aligned(16))) float smem[];
  constexpr int KST = BN == 16 ? 16 : BN + 16;   // conv_lds_kst
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int slot = a.slot0 + (int)blockIdx.y;
  const int n0 = (int)blockIdx.z * BN;
  const int Mslot = a.nx * a.P;                  // < 2^31 (checked by the launcher)
  const int Hp2 = a.H + 2 * a.pad, Wp2 = a.W + 2 * a.pad;
  const int img = Hp2 * Wp2 * a.C;
  const bool virt = a.vin.chmap != nullptr;
  float* imgs = smem;
  float* Ws = imgs + (int64_t)nimg_cap * img;    // [kpad + 8][KST], k-major, zero padded
  int* koff = reinterpret_cast<int*>(Ws + KST * (kpad + 8));   // [kpad + 16]
  int* chrow = koff + kpad + 16;
  const float* __restrict__ X = reinterpret_cast<const float*>(a.in.p);
  const float* __restrict__ bias = a.btab[slot];
  const float* __restrict__ cache = reinterpret_cast<const float*>(a.vin.cache);
  const float* __restrict__ delta = reinterpret_cast<const float*>(a.vin.delta);

  const int ncol = a.cols ? a.ncols : a.Cout;
  __shared__ const float* wrow[BN];      // weight row of each column (nullptr: none)
  __shared__ uint64_t chmask_s;          // input channels the mutant's map changes
  if (tid < BN) {
    const int n = n0 + tid;
    const float* wr = nullptr;
    if (n < ncol) {
      if (a.cols) {
        const DeltaCol cd = a.cols[n];
        wr = reinterpret_cast<const float*>(a.wtab[a.slot0 + cd.slot - a.col_slot0]) + (int64_t)cd.c * a.K;
      } else {
        wr = reinterpret_cast<const float*>(a.wtab[slot]) + (int64_t)n * a.K;
      }
    }
    wrow[tid] = wr;
  }
  for (int k = tid; k < kpad + 16; k += 256) {
    int o = 0;
    if (k < a.K) {
      const int ci = k % a.C, t = k / a.C;
      o = ((t / a.kw) * Wp2 + (t % a.kw)) * a.C + ci;
    }
    koff[k] = 4 * o;                     // bytes
  }
  if (virt) {
    for (int c = tid; c < a.C; c += 256) chrow[c] = a.vin.chmap[(int64_t)slot * a.C + c];
    __syncthreads();
    if (wave == 0) {
      const uint64_t m = __ballot(lane < a.C && chrow[lane] != lane);
      if (lane == 0) chmask_s = m;
    }
  }
  __syncthreads();
  // weights, k-major: eight loads per thread in flight, then their writes
  {
    typedef __attribute__((address_space(1))) const float gfloat;
    const int nw = (kpad + 8) * BN;
    for (int e0 = tid; e0 < nw; e0 += 256 * 8) {
      float wv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = e0 + 256 * u, k = e / BN, n = e % BN;
        const float* wr = e < nw ? wrow[n] : nullptr;
        wv[u] = (wr != nullptr && k < a.K) ? ((const gfloat*)wr)[k] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = e0 + 256 * u;
        if (e < nw) {
          const int k = e / BN, n = e % BN;
          Ws[PAIR ? ((k >> 1) * KST + n) * 2 + (k & 1) : k * KST + n] = wv[u];
        }
      }
    }
  }
  const uint64_t chmask = virt ? chmask_s : 0;

  // per piece: the image offset of each GEMM row's receptive field, and the
  // output offset of each group of 4 rows (a pool window, or 4 pixels)
  __shared__ int rowbase[256];
  __shared__ int64_t grpout[64];
  const bool grp_ok = !a.cols && (a.pool || a.P % 4 == 0);
  constexpr int TN = BN / 16;
  // per column of this lane: bias, output slot, channel offset and stride
  float bv[TN];
  int oslot[TN], ochan[TN];
  const int ostride = a.cols && a.delta_T > 0 ? a.delta_T : a.Cout;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int n = n0 + j * 16 + (lane & 15);
    bv[j] = 0.f;
    oslot[j] = slot;
    ochan[j] = n;
    if (n < ncol) {
      if (a.cols) {
        const DeltaCol cd = a.cols[n];
        bv[j] = a.btab[a.slot0 + cd.slot - a.col_slot0][cd.c];
        oslot[j] = a.slot0 + cd.slot - a.col_slot0;
        ochan[j] = a.delta_T > 0 ? cd.t : cd.c;
      } else {
        bv[j] = bias[n];
      }
    }
    // complete these loads here: left pending into the piece loop, every
    // use in the epilogue would wait for all outstanding memory operations
    asm volatile("" ::"v"(bv[j]), "v"(oslot[j]), "v"(ochan[j]));
  }

  // A piece is 256 GEMM rows; its images are staged in LDS.  When they fit in
  // NPF 16-byte registers per thread and need no padding, every load of a
  // piece (and a virtual input's values for up to NFC changed channels of
  // NPX pixels per thread) is issued before the first LDS write, so staging
  // costs one memory round trip; the registers are free again before the k
  // loop, which keeps the block's register budget at the k loop's.
  constexpr int NPF = 5, NPX = 4, NFC = 2;
  const int nfc = __popcll(chmask);
  const bool pre = a.pad == 0 && (img & 3) == 0 && nimg_cap * img <= 1024 * NPF &&
                   (virt ? a.C <= 64 && nfc <= NFC && nimg_cap * a.H * a.W <= 256 * NPX
                         : a.in.row_elems == img);
  int fc[NFC], fs[NFC];                // changed channels and their map entries
  {
    uint64_t m = chmask;
#pragma unroll
    for (int q = 0; q < NFC; ++q) {
      fc[q] = m ? __builtin_ctzll(m) : 0;
      fs[q] = m ? chrow[fc[q]] : 0;
      m &= m - 1;
    }
  }
  auto piece = [&](int it, int& xf, int& ni) -> bool {
    if (it >= iters) return false;
    const int m0 = ((int)blockIdx.x * iters + it) * 256;
    if (m0 >= Mslot) return false;
    xf = (int)divu(a.dP, (uint32_t)m0);
    ni = min(a.nx - 1, (int)divu(a.dP, (uint32_t)(m0 + 255))) - xf + 1;
    return true;
  };
  // rows of one piece are consecutive in both tensor modes
  auto src_of = [&](int xf) {
    return virt ? cache + ((int64_t)a.x0 + xf) * img
                : X + row_index(a.in.mode, (int64_t)slot * a.nx + xf, a.nx, a.x0) * a.in.row_elems;
  };
  // the piece's images: all loads first, then their 16-byte LDS writes, then
  // (after a barrier) the changed channels of a virtual input, again loads first
  // tz: the thread index through a move the compiler cannot see through, so
  // the index arithmetic stays inside each call instead of being hoisted out
  // of the piece loop and held in registers across the k loop
  auto put = [&](int xf, int ni) {
    int tz;
    asm volatile("v_mov_b32 %0, %1" : "=v"(tz) : "v"(tid));
    const float* src = src_of(xf);
    const int nv = ni * img / 4;
    {
      v4f pf[NPF] = {};
#pragma unroll
      for (int u = 0; u < NPF; ++u) {
        const int e4 = tz + 256 * u;
        if (e4 < nv) pf[u] = *reinterpret_cast<const v4f*>(src + 4 * e4);
      }
      v4f* dst = reinterpret_cast<v4f*>(imgs);
#pragma unroll
      for (int u = 0; u < NPF; ++u) {
        const int e4 = tz + 256 * u;
        if (e4 < nv) dst[e4] = pf[u];
      }
    }
    if (nfc) {
      const int HW = a.H * a.W;
      float fx[NPX][NFC] = {};
#pragma unroll
      for (int w = 0; w < NPX; ++w) {
        const int e = tz + 256 * w;
        int ii, pix;
        divmodu(a.dHW, (uint32_t)e, ii, pix);
        if (e >= ni * HW) continue;
#pragma unroll
        for (int q = 0; q < NFC; ++q) {
          const int sq = fs[q];
          if (q < nfc && sq != -1)
            fx[w][q] = sq >= 0 ? src[(int64_t)e * a.C + sq]
                     : delta[(((int64_t)slot * a.nx + xf + ii) * HW + pix) * a.vin.T + (-2 - sq)];
        }
      }
      __syncthreads();                 // the 16-byte writes land first
#pragma unroll
      for (int w = 0; w < NPX; ++w) {
        const int e = tz + 256 * w;
        if (e >= ni * HW) continue;
#pragma unroll
        for (int q = 0; q < NFC; ++q)
          if (q < nfc) imgs[e * a.C + fc[q]] = fx[w][q];
      }
    }
  };
  // images of one piece without registers in between (padding, or too big)
  auto stage = [&](int xi_first, int nimg) {
    if (a.pad == 0 && (img & 3) == 0 && (virt ? a.C <= 64 : a.in.row_elems == img)) {
      // 16-byte copies of the rows (a virtual input's cached original
      // images), then the channels the mutant's map changes
      const float* src = virt ? cache + ((int64_t)a.x0 + xi_first) * img
                              : X + row_index(a.in.mode, (int64_t)slot * a.nx + xi_first, a.nx, a.x0) * a.in.row_elems;
      const v4f* src4 = reinterpret_cast<const v4f*>(src);
      v4f* dst = reinterpret_cast<v4f*>(imgs);
      for (int e = tid; e < nimg * img / 4; e += 256) dst[e] = src4[e];
      if (chmask) {
        __syncthreads();
        const int HW = a.H * a.W;
        for (int e = tid; e < nimg * HW; e += 256) {
          int ii, pix;
          divmodu(a.dHW, (uint32_t)e, ii, pix);
          const float* cp = src + (int64_t)e * a.C;
          const float* dp = delta + (((int64_t)slot * a.nx + xi_first + ii) * HW + pix) * a.vin.T;
          for (uint64_t m = chmask; m; m &= m - 1) {
            const int c = __builtin_ctzll(m), s = chrow[c];
            imgs[e * a.C + c] = s >= 0 ? cp[s] : s == -1 ? 0.f : dp[-2 - s];
          }
        }
      }
      return;
    }
    for (int e = tid; e < nimg * img; e += 256) {
      const int ii = e / img, rem = e % img;
      const int c = rem % a.C, pix = rem / a.C;
      const int iy = pix / Wp2 - a.pad, ix = pix % Wp2 - a.pad;
      float v = 0.f;
      if (iy >= 0 && iy < a.H && ix >= 0 && ix < a.W) {
        const int xi = xi_first + ii;
        const int64_t r = (int64_t)slot * a.nx + xi;
        if (virt) {
          v = virtual_elem<float>(a.vin, chrow, r, xi, a.x0, iy * a.W + ix, c);
        } else {
          v = X[row_index(a.in.mode, r, a.nx, a.x0) * a.in.row_elems + ((int64_t)iy * a.W + ix) * a.C + c];
        }
      }
      imgs[e] = v;
    }
  };

  v4f acc[4][TN];
  auto epilogue = [&](int m0) {
    const int mw = m0 + wave * 64;
    if (grp_ok) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int mb = mw + i * 16 + (lane >> 4) * 4;
        if (mb >= Mslot) continue;
        const int64_t go = grpout[(wave * 64 + i * 16 + (lane >> 4) * 4) >> 2];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int n = n0 + j * 16 + (lane & 15);
          if (n >= ncol) continue;
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = act(acc[i][j][e] + bv[j], a.relu);
          if (a.pool) {
            store_out<float>(a.out, a.out_f32, go + n, fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3])));
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) store_out<float>(a.out, a.out_f32, go + (int64_t)e * a.Cout + n, v[e]);
          }
        }
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int mb = mw + i * 16 + (lane >> 4) * 4;
      if (mb >= Mslot) continue;
      int xo, pb;
      divmodu(a.dP, (uint32_t)mb, xo, pb);
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int n = n0 + j * 16 + (lane & 15);
        if (n >= ncol) continue;
        const int64_t ro = row_index(a.out_mode, (int64_t)oslot[j] * a.nx + xo, a.nx, a.x0);
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[e] = acc[i][j][e] + bv[j];
          v[e] = act(v[e], a.relu);
        }
        if (a.pool) {
          const float mx = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
          store_out<float>(a.out, a.out_f32, ro * a.out_row + (int64_t)(pb >> 2) * ostride + ochan[j], mx);
        } else {
          // the lane's 4 rows may cross into the next input when P % 4 != 0
          int xe = xo, pe = pb;
          int64_t re = ro;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (mb + e >= Mslot) break;
            if (pe == a.P) {
              ++xe; pe = 0;
              re = row_index(a.out_mode, (int64_t)oslot[j] * a.nx + xe, a.nx, a.x0);
            }
            store_out<float>(a.out, a.out_f32, re * a.out_row + (int64_t)pe * ostride + ochan[j], v[e]);
            ++pe;
          }
        }
      }
    }
  };

  int xf = 0, ni = 0;
  bool have = piece(0, xf, ni);
  for (int it = 0; have; ++it) {
    const int m0 = ((int)blockIdx.x * iters + it) * 256;
    const int xi_first = xf, nimg = ni;
    __syncthreads();                   // previous piece done with imgs and rowbase
    if (pre) {
      put(xi_first, nimg);
    } else {
      stage(xi_first, nimg);
    }
    {
      const int m = m0 + tid;
      int b = 0;
      if (m < Mslot) {
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
        b = (xi - xi_first) * img + (oy * a.stride * Wp2 + ox * a.stride) * a.C;
        if (grp_ok && (tid & 3) == 0) {
          const int64_t ro = a.out_mode == MODE_BUF ? (int64_t)slot * a.nx + xi : (int64_t)a.x0 + xi;
          grpout[tid >> 2] = ro * a.out_row + (int64_t)(a.pool ? (p >> 2) : p) * a.Cout;
        }
      }
      rowbase[tid] = b;
    }
    __syncthreads();
    // row offsets in bytes, with the LDS address of the images folded in
    const char* imgb = reinterpret_cast<const char*>(imgs);
    int base[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) base[i] = 4 * rowbase[wave * 64 + i * 16 + (lane & 15)];
    have = piece(it + 1, xf, ni);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};
    // software pipeline over steps of 8 k with two register sets: the reads
    // of step s + 1 are issued before the MFMAs of step s, and the offsets
    // of step s + 2 before those (the padded table rows past kpad are zero)
    int k8 = 0;
    if constexpr (PAIR) {
      const float* wl = Ws + ((lane >> 4) * KST + (lane & 15)) * 2;
      const int* kl = koff + 2 * (lane >> 4);
      v2f a0[4], b0[TN], a1[4], b1[TN];
      int ko;
#define MURE_LDS_READ(A, B, KB, O)                                              \
      _Pragma("unroll") for (int i = 0; i < 4; ++i)                            \
        A[i] = *reinterpret_cast<const v2f*>(imgb + base[i] + (O));            \
      _Pragma("unroll") for (int j = 0; j < TN; ++j)                           \
        B[j] = *reinterpret_cast<const v2f*>(wl + ((KB) / 2 * KST + j * 16) * 2);
#define MURE_LDS_MFMA(A, B)                                                    \
      _Pragma("unroll") for (int h = 0; h < 2; ++h)                            \
      _Pragma("unroll") for (int i = 0; i < 4; ++i)                            \
      _Pragma("unroll") for (int j = 0; j < TN; ++j)                           \
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(A[i][h], B[j][h], acc[i][j], 0, 0, 0);
      MURE_LDS_READ(a0, b0, 0, kl[0])
      ko = kl[8];
      for (; k8 + 16 <= kpad; k8 += 16) {
        MURE_LDS_READ(a1, b1, k8 + 8, ko)
        ko = kl[k8 + 16];
        __builtin_amdgcn_sched_barrier(0);
        MURE_LDS_MFMA(a0, b0)
        __builtin_amdgcn_sched_barrier(0);
        MURE_LDS_READ(a0, b0, k8 + 16, ko)
        ko = kl[k8 + 24];
        __builtin_amdgcn_sched_barrier(0);
        MURE_LDS_MFMA(a1, b1)
        __builtin_amdgcn_sched_barrier(0);
      }
      if (k8 < kpad) { MURE_LDS_MFMA(a0, b0) }      // kpad % 16 == 8: the last step
#undef MURE_LDS_READ
#undef MURE_LDS_MFMA
    } else {
      const float* wl = Ws + (lane >> 4) * KST + (lane & 15);
      const int* kl = koff + (lane >> 4);
      float a0[2][4], b0[2][TN], a1[2][4], b1[2][TN];
      int ko[2];
#define MURE_LDS_READ(A, B, KB, O0, O1)                                         \
      _Pragma("unroll") for (int i = 0; i < 4; ++i) {                          \
        A[0][i] = *reinterpret_cast<const float*>(imgb + base[i] + (O0));      \
        A[1][i] = *reinterpret_cast<const float*>(imgb + base[i] + (O1));      \
      }                                                                        \
      _Pragma("unroll") for (int j = 0; j < TN; ++j) {                         \
        B[0][j] = wl[(KB) * KST + j * 16];                                     \
        B[1][j] = wl[((KB) + 4) * KST + j * 16];                               \
      }
#define MURE_LDS_MFMA(A, B)                                                    \
      _Pragma("unroll") for (int h = 0; h < 2; ++h)                            \
      _Pragma("unroll") for (int i = 0; i < 4; ++i)                            \
      _Pragma("unroll") for (int j = 0; j < TN; ++j)                           \
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(A[h][i], B[h][j], acc[i][j], 0, 0, 0);
      MURE_LDS_READ(a0, b0, 0, kl[0], kl[4])
      ko[0] = kl[8];
      ko[1] = kl[12];
      for (; k8 + 16 <= kpad; k8 += 16) {
        MURE_LDS_READ(a1, b1, k8 + 8, ko[0], ko[1])
        ko[0] = kl[k8 + 16];
        ko[1] = kl[k8 + 20];
        __builtin_amdgcn_sched_barrier(0);
        MURE_LDS_MFMA(a0, b0)
        __builtin_amdgcn_sched_barrier(0);
        MURE_LDS_READ(a0, b0, k8 + 16, ko[0], ko[1])
        ko[0] = kl[k8 + 24];
        ko[1] = kl[k8 + 28];
        __builtin_amdgcn_sched_barrier(0);
        MURE_LDS_MFMA(a1, b1)
        __builtin_amdgcn_sched_barrier(0);
      }
      if (k8 < kpad) { MURE_LDS_MFMA(a0, b0) }      // kpad % 16 == 8: the last step
#undef MURE_LDS_READ
#undef MURE_LDS_MFMA
    }
    epilogue(m0);
  }
}

hipError_t launch_conv_lds(const ConvArgs& a0, int nslots, hipStream_t s) {
  if (nslots <= 0 || a0.nx <= 0) return hipSuccess;
  if ((int64_t)a0.nx * a0.P + 256 >= INT32_MAX) return hipErrorInvalidValue;
  if (a0.pool && a0.P % 4) return hipErrorInvalidValue;
  if (a0.cols && (a0.vin.chmap || a0.in.mode != MODE_CACHE || a0.ncols <= 0)) return hipErrorInvalidValue;
  if (!a0.cols && a0.Cout > 64) return hipErrorInvalidValue;
  ConvArgs a = a0;
  a.dP = make_divu32((uint32_t)a.P);
  a.dWp = make_divu32((uint32_t)std::max(1, a.Wp));
  a.dWc = make_divu32((uint32_t)std::max(1, a.Wc));
  a.dHW = make_divu32((uint32_t)std::max(1, a.H * a.W));
  a.dC = make_divu32((uint32_t)std::max(1, a.C));
  a.dImg = make_divu32((uint32_t)std::max(1, (a.H + 2 * a.pad) * (a.W + 2 * a.pad) * a.C));
  // columns per block: the node's channels, or for a gathered delta the
  // widest tile whose LDS fits
  int bn = conv_lds_bn(a.Cout);
  size_t lds = (size_t)conv_lds_bytes(a.H, a.W, a.C, a.pad, a.P, a.Cout, a.K);
  if (a.cols) {
    for (bn = conv_lds_bn(std::min(a.ncols, 64)); bn > 16; bn /= 2)
      if (conv_lds_bytes(a.H, a.W, a.C, a.pad, a.P, bn, a.K) <= 64 * 1024) break;
    lds = (size_t)conv_lds_bytes(a.H, a.W, a.C, a.pad, a.P, bn, a.K);
    nslots = 1;
  }
  const int kpad = (a.K + 7) / 8 * 8;
  const int cap = conv_lds_nimg_cap(a.P);
  if (lds > 64 * 1024) return hipErrorInvalidValue;
  const int64_t Mslot = (int64_t)a.nx * a.P;
  const int64_t pieces = (Mslot + 255) / 256;
  const int ncol = a.cols ? a.ncols : a.Cout;
  const int64_t ztiles = (ncol + bn - 1) / bn;
  // about 2048 blocks in flight, at most 8 pieces per block
  int iters = (int)std::max<int64_t>(1, std::min<int64_t>(8, pieces * nslots * ztiles / 2048));
  dim3 grid((unsigned)((pieces + iters - 1) / iters), (unsigned)nslots, (unsigned)ztiles);
  const bool pair = a.C % 2 == 0;
  switch (bn * 2 + (pair ? 1 : 0)) {
    case 32: hipLaunchKernelGGL((conv_lds_kernel<16, false>), grid, dim3(256), lds, s, a, cap, kpad, iters); break;
    case 33: hipLaunchKernelGGL((conv_lds_kernel<16, true>), grid, dim3(256), lds, s, a, cap, kpad, iters); break;
    case 64: hipLaunchKernelGGL((conv_lds_kernel<32, false>), grid, dim3(256), lds, s, a, cap, kpad, iters); break;
    case 65: hipLaunchKernelGGL((conv_lds_kernel<32, true>), grid, dim3(256), lds, s, a, cap, kpad, iters); break;
    case 128: hipLaunchKernelGGL((conv_lds_kernel<64, false>), grid, dim3(256), lds, s, a, cap, kpad, iters); break;
    default: hipLaunchKernelGGL((conv_lds_kernel<64, true>), grid, dim3(256), lds, s, a, cap, kpad, iters); break;
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------- VALU conv
// SPEC = 1: 5x5 kernel, one input channel, stride 1, 2x2 pooling (LeNet's
// first layer): the 6x6 input patch of a pooling window sits in registers.
template <typename T, int SPEC>
__global__ __launch_bounds__(256) void conv_valu_kernel(ValuArgs a, int R) {
  extern __shared__ __attribute__((aligned(16))) float vsm[];
  const int tid = threadIdx.x;
  const int sl = a.slot0 + (int)blockIdx.y;
  const int xi0 = (int)blockIdx.x * R;
  const int nr = min(R, a.nx - xi0);
  const int Q = a.Hp * a.Wp;
  const int Hp2 = a.H + 2 * a.pad, Wp2 = a.W + 2 * a.pad;
  const int img = Hp2 * Wp2 * a.C;
  int c_beg = 0, c_end = a.Cout;
  if (a.ch_off) { c_beg = a.ch_off[sl]; c_end = a.ch_off[sl + 1]; }
  const int nall = c_end - c_beg;
  if (nall <= 0 || nr <= 0) return;
  float* imgs = vsm;
  float* Wl = imgs + (int64_t)R * img;                 // [nall][K]
  const T* __restrict__ Wt = reinterpret_cast<const T*>(a.wtab[sl]);
  const float* __restrict__ bias = a.btab[sl];
  for (int e = tid; e < nall * a.K; e += 256) {
    const int u = e / a.K, k = e - u * a.K;
    const int c = a.ch_list ? a.ch_list[c_beg + u] : c_beg + u;
    Wl[e] = to_f<T>(Wt[(int64_t)c * a.K + k]);
  }
  const T* __restrict__ X = reinterpret_cast<const T*>(a.in.p);
  if (a.pad == 0 && a.in.row_elems == img) {
    // rows of one launch are consecutive in both tensor modes
    const T* src = X + row_index(a.in.mode, (int64_t)sl * a.nx + xi0, a.nx, a.x0) * a.in.row_elems;
    for (int e = tid; e < nr * img; e += 256) imgs[e] = to_f<T>(src[e]);
  } else {
    for (int e = tid; e < nr * img; e += 256) {
      const int ii = e / img, rem = e - ii * img;
      const int c = rem % a.C, pix = rem / a.C;
      const int iy = pix / Wp2 - a.pad, ix = pix % Wp2 - a.pad;
      float v = 0.f;
      if (iy >= 0 && iy < a.H && ix >= 0 && ix < a.W) {
        const int64_t ri = row_index(a.in.mode, (int64_t)sl * a.nx + xi0 + ii, a.nx, a.x0);
        v = to_f<T>(X[ri * a.in.row_elems + ((int64_t)iy * a.W + ix) * a.C + c]);
      }
      imgs[e] = v;
    }
  }
  __syncthreads();
  const int npix = a.pool ? 4 : 1;
  const float invWp = 1.0f / (float)a.Wp;
  int rr = tid / Q, q = tid - (tid / Q) * Q;
  for (int p = tid; p < nr * Q; p += 256) {
    const float* im = imgs + (int64_t)rr * img;
    int qy, qx;
    fast_divmod(q, a.Wp, invWp, qy, qx);
    const int64_t r = (int64_t)sl * a.nx + xi0 + rr;
    const int64_t ro = row_index(a.out_mode, r, a.nx, a.x0);
    if constexpr (SPEC == 1) {
      float pt[6][6];
      const float* p0 = im + (2 * qy) * Wp2 + 2 * qx;
#pragma unroll
      for (int y = 0; y < 6; ++y)
#pragma unroll
        for (int x = 0; x < 6; ++x) pt[y][x] = p0[y * Wp2 + x];
      for (int u = 0; u < nall; ++u) {
        const float* wu = Wl + u * 25;
        float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
        for (int dy = 0; dy < 5; ++dy)
#pragma unroll
          for (int dx = 0; dx < 5; ++dx) {
            const float w = wu[dy * 5 + dx];
            a0 = fmaf(pt[dy][dx], w, a0);
            a1 = fmaf(pt[dy][dx + 1], w, a1);
            a2 = fmaf(pt[dy + 1][dx], w, a2);
            a3 = fmaf(pt[dy + 1][dx + 1], w, a3);
          }
        const int c = a.ch_list ? a.ch_list[c_beg + u] : c_beg + u;
        const float bv = bias[c];
        float v0 = a0 + bv, v1 = a1 + bv, v2 = a2 + bv, v3 = a3 + bv;
        v0 = act(v0, a.relu); v1 = act(v1, a.relu); v2 = act(v2, a.relu); v3 = act(v3, a.relu);
        const float v = fmaxf(fmaxf(v0, v1), fmaxf(v2, v3));
        if (a.delta_T > 0) store_out<T>(a.out, 0, ro * a.out_row + (int64_t)q * a.delta_T + u, v);
        else store_out<T>(a.out, a.out_f32, ro * a.out_row + (int64_t)q * a.Cout + c, v);
      }
    } else {
      int off[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int oy, ox;
        if (a.pool) { oy = 2 * qy + (j >> 1); ox = 2 * qx + (j & 1); }
        else { oy = qy; ox = qx; }
        off[j] = (oy * a.stride * Wp2 + ox * a.stride) * a.C;
      }
      for (int ub = 0; ub < nall; ub += 8) {
        const int nch = min(8, nall - ub);
        float acc[4][8];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int u = 0; u < 8; ++u) acc[j][u] = 0.f;
        int k = 0;
        for (int dy = 0; dy < a.kh; ++dy)
          for (int dx = 0; dx < a.kw; ++dx) {
            const int tap = (dy * Wp2 + dx) * a.C;
            for (int ci = 0; ci < a.C; ++ci, ++k) {
              float xv[4];
#pragma unroll
              for (int j = 0; j < 4; ++j) xv[j] = j < npix ? im[off[j] + tap + ci] : 0.f;
#pragma unroll
              for (int u = 0; u < 8; ++u) {
                if (u >= nch) break;
                const float w = Wl[(ub + u) * a.K + k];
#pragma unroll
                for (int j = 0; j < 4; ++j)
                  if (j < npix) acc[j][u] = fmaf(xv[j], w, acc[j][u]);
              }
            }
          }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (u >= nch) break;
          const int c = a.ch_list ? a.ch_list[c_beg + ub + u] : c_beg + ub + u;
          const float bv = bias[c];
          float v = acc[0][u] + bv;
          v = act(v, a.relu);
          for (int j = 1; j < npix; ++j) {
            float w2 = acc[j][u] + bv;
            w2 = act(w2, a.relu);
            v = fmaxf(v, w2);
          }
          if (a.delta_T > 0)
            store_out<T>(a.out, 0, ro * a.out_row + (int64_t)q * a.delta_T + ub + u, v);
          else
            store_out<T>(a.out, a.out_f32, ro * a.out_row + (int64_t)q * a.Cout + c, v);
        }
      }
    }
    q += 256;
    while (q >= Q) { q -= Q; ++rr; }
  }
}

// The delta of LeNet's first layer (5x5, one input channel, 2x2 pooling) over
// the shared cached input: a block stages its R images once and computes the
// listed channels of a group of up to SPB slots from them (the image patch of
// a pooling window stays in registers across every slot and channel).  Each
// output's chain is the SPEC = 1 kernel's, so results are bit-identical.
constexpr int VALU_SPB = 32;
template <typename T>
__global__ __launch_bounds__(256) void conv_valu_slots_kernel(ValuArgs a, int R) {
  extern __shared__ __attribute__((aligned(16))) float vsm[];
  const int tid = threadIdx.x;
  const int xi0 = (int)blockIdx.x * R;
  const int nr = min(R, a.nx - xi0);
  const int s_beg = a.slot0 + (int)blockIdx.y * VALU_SPB;
  const int s_end = min(a.slot0 + a.nslots, s_beg + VALU_SPB);
  const int u_beg = a.ch_off[s_beg], u_end = a.ch_off[s_end];
  if (nr <= 0 || u_end <= u_beg) return;
  const int Q = a.Hp * a.Wp;
  const int Wp2 = a.W, img = a.H * a.W;                // no padding, one input channel
  float* imgs = vsm;
  float* Wl = imgs + (int64_t)R * img;                 // [u - u_beg][25]
  for (int sl = s_beg; sl < s_end; ++sl) {
    const T* __restrict__ Wt = reinterpret_cast<const T*>(a.wtab[sl]);
    for (int e = tid; e < (a.ch_off[sl + 1] - a.ch_off[sl]) * 25; e += 256) {
      const int u = a.ch_off[sl] + e / 25, k = e % 25;
      Wl[(u - u_beg) * 25 + k] = to_f<T>(Wt[(int64_t)a.ch_list[u] * 25 + k]);
    }
  }
  // the images are the prefix cache's rows x0 + xi0 .. (shared by every slot)
  const T* src = reinterpret_cast<const T*>(a.in.p) + ((int64_t)a.x0 + xi0) * a.in.row_elems;
  for (int e = tid; e < nr * img; e += 256) imgs[e] = to_f<T>(src[e]);
  __syncthreads();
  const float invWp = 1.0f / (float)a.Wp;
  for (int p = tid; p < nr * Q; p += 256) {
    const int rr = p / Q, q = p - rr * Q;
    int qy, qx;
    fast_divmod(q, a.Wp, invWp, qy, qx);
    float pt[6][6];
    const float* p0 = imgs + (int64_t)rr * img + (2 * qy) * Wp2 + 2 * qx;
#pragma unroll
    for (int y = 0; y < 6; ++y)
#pragma unroll
      for (int x = 0; x < 6; ++x) pt[y][x] = p0[y * Wp2 + x];
    for (int sl = s_beg; sl < s_end; ++sl) {
      const int c_beg = a.ch_off[sl], c_end = a.ch_off[sl + 1];
      if (c_end <= c_beg) continue;
      const float* __restrict__ bias = a.btab[sl];
      const int64_t ro = row_index(a.out_mode, (int64_t)sl * a.nx + xi0 + rr, a.nx, a.x0);
      for (int u = c_beg; u < c_end; ++u) {
        const float* wu = Wl + (u - u_beg) * 25;
        float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
        for (int dy = 0; dy < 5; ++dy)
#pragma unroll
          for (int dx = 0; dx < 5; ++dx) {
            const float w = wu[dy * 5 + dx];
            a0 = fmaf(pt[dy][dx], w, a0);
            a1 = fmaf(pt[dy][dx + 1], w, a1);
            a2 = fmaf(pt[dy + 1][dx], w, a2);
            a3 = fmaf(pt[dy + 1][dx + 1], w, a3);
          }
        const int c = a.ch_list[u];
        const float bv = bias[c];
        float v0 = a0 + bv, v1 = a1 + bv, v2 = a2 + bv, v3 = a3 + bv;
        v0 = act(v0, a.relu); v1 = act(v1, a.relu); v2 = act(v2, a.relu); v3 = act(v3, a.relu);
        const float v = fmaxf(fmaxf(v0, v1), fmaxf(v2, v3));
        if (a.delta_T > 0) store_out<T>(a.out, 0, ro * a.out_row + (int64_t)q * a.delta_T + (u - c_beg), v);
        else store_out<T>(a.out, a.out_f32, ro * a.out_row + (int64_t)q * a.Cout + c, v);
      }
    }
  }
}

hipError_t launch_valu(const ValuArgs& a, int dtype, hipStream_t s) {
  if (a.nslots <= 0 || a.nx <= 0) return hipSuccess;
  const int Q = a.Hp * a.Wp;
  const int R = valu_rows(Q);
  const size_t lds = (size_t)valu_lds_bytes(a.H, a.W, a.C, a.pad, Q, a.Cout, a.K);
  if (lds > 64 * 1024) return hipErrorInvalidValue;
  dim3 grid((unsigned)((a.nx + R - 1) / R), (unsigned)a.nslots);
  const bool spec = a.kh == 5 && a.kw == 5 && a.C == 1 && a.stride == 1 && a.pool;
  if (spec && a.ch_off && a.ch_list && a.in.mode == MODE_CACHE && a.pad == 0 && a.in.row_elems == a.H * a.W &&
      !a.out_f32) {
    // channel lists over the shared cached input: slot groups share staged
    // images.  A slot lists at most delta_T channels when it writes compact
    // delta rows, so the weight section holds VALU_SPB * min(C_out, delta_T)
    // channels; with at most 4 images per block the LDS stays near 22 KB
    // and seven blocks share a CU (the FMA chains wait on LDS and global
    // latency, which more resident waves hide)
    const int cmax = a.delta_T > 0 ? std::min(a.Cout, a.delta_T) : a.Cout;
    const int R2 = std::min(R, 4);
    const size_t lds2 = ((size_t)R2 * a.H * a.W + (size_t)VALU_SPB * cmax * 25) * sizeof(float);
    if (lds2 <= 64 * 1024) {
      dim3 g2((unsigned)((a.nx + R2 - 1) / R2), (unsigned)((a.nslots + VALU_SPB - 1) / VALU_SPB));
      if (dtype == 0) hipLaunchKernelGGL(conv_valu_slots_kernel<float>, g2, dim3(256), lds2, s, a, R2);
      else hipLaunchKernelGGL(conv_valu_slots_kernel<bf16_t>, g2, dim3(256), lds2, s, a, R2);
      return hipGetLastError();
    }
  }
  if (dtype == 0) {
    if (spec) hipLaunchKernelGGL((conv_valu_kernel<float, 1>), grid, dim3(256), lds, s, a, R);
    else hipLaunchKernelGGL((conv_valu_kernel<float, 0>), grid, dim3(256), lds, s, a, R);
  } else {
    if (spec) hipLaunchKernelGGL((conv_valu_kernel<bf16_t, 1>), grid, dim3(256), lds, s, a, R);
    else hipLaunchKernelGGL((conv_valu_kernel<bf16_t, 0>), grid, dim3(256), lds, s, a, R);
  }
  return hipGetLastError();
}

}  // namespace mure
