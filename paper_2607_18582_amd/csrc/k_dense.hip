// DENSE layers as a GEMM on MFMA (gfx950), optionally fused with the kill
// reduction of the network output.
//
// Rows are (mutant slot, input) pairs; a block owns 64 consecutive inputs of
// one slot and BN output units, so with the kill fused one wavefront turns the
// block's 64 rows into one 64-bit kill word.  The reduction over k runs in
// increasing steps of the MFMA's depth (4 for fp32, 32 for bf16), the same
// order as every other kernel computing the node.
#include <climits>

#include "dev.hpp"

namespace mure {

template <typename T> struct DenseCfg;
template <> struct DenseCfg<float> { static constexpr int BK = 32, VEC = 4, PAD = 4; };
template <> struct DenseCfg<bf16_t> { static constexpr int BK = 64, VEC = 8, PAD = 8; };

// VIRT: the input is the first mutated node's output seen through the
// mutant's channel map: a per-block table maps each k of the flattened row to
// the cached original, zero, or a compact delta entry.
//
// The next k chunk's global loads are issued into registers before the MFMAs
// of the current chunk (register prefetch); tiles are staged as raw 16-byte
// vectors.
// BM: rows (inputs) per block; 64 whenever the kill is fused (one wave's
// ballot is one kill word).
template <typename T, int BN, int WAVES_M, bool VIRT, int BM>
__global__ __launch_bounds__(256) void dense_kernel(DenseArgs a) {
  constexpr int BK = DenseCfg<T>::BK, VEC = DenseCfg<T>::VEC, LD = BK + DenseCfg<T>::PAD;
  constexpr int WAVES_N = 4 / WAVES_M;
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int LSN = BN <= 64 ? BM * (BN + 1) : 1;
  constexpr int KV = BK / VEC;                               // 16-byte vectors per tile row
  constexpr int APT = BM * KV / 256;                         // A vectors per thread
  constexpr int BPT = (BN * KV + 255) / 256;                 // B vectors per thread
  __shared__ __attribute__((aligned(16))) T As[BM * LD];
  __shared__ __attribute__((aligned(16))) T Bs[BN * LD];
  __shared__ float Ls[LSN];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  const int slot = a.slot0 + (int)blockIdx.y;
  const int m0 = (int)blockIdx.x * BM;
  const int n0 = (int)blockIdx.z * BN;
  const T* __restrict__ Wt = reinterpret_cast<const T*>(a.wtab[slot]);
  const T* __restrict__ X = reinterpret_cast<const T*>(a.in.p);
  const int ncol = a.cols ? a.ncols : a.Cout;
  // the weight row of each column of the block (a gathered delta takes each
  // column's row from its own mutant's weights); nullptr past the last column
  __shared__ const T* wrow[BN];
  for (int n = tid; n < BN; n += 256) {
    const T* w = nullptr;
    if (n0 + n < ncol) {
      if (a.cols) {
        const DeltaCol cd = a.cols[n0 + n];
        w = reinterpret_cast<const T*>(a.wtab[a.slot0 + cd.slot - a.col_slot0]) + (int64_t)cd.c * a.K;
      } else {
        w = Wt + (int64_t)(n0 + n) * a.K;
      }
    }
    wrow[n] = w;
  }

  // VIRT: the k map (K ints) and per-vector identity flags (K / VEC bytes) in
  // dynamic LDS sized to the layer
  extern __shared__ __attribute__((aligned(16))) int dense_dyn[];
  int* const kmap = dense_dyn;
  unsigned char* const kdirect = reinterpret_cast<unsigned char*>(dense_dyn + (VIRT ? a.K : 0));
  if constexpr (VIRT) {
    const int32_t* chrow = a.vin.chmap + (int64_t)slot * a.vin.C;
    for (int k = tid; k < a.K; k += 256) {
      const int pix = k / a.vin.C, c = k - pix * a.vin.C;
      const int src = chrow[c];
      kmap[k] = src >= 0 ? pix * a.vin.C + src
              : src == -1 ? INT_MIN : -1 - (pix * a.vin.T + (-2 - src));
    }
    __syncthreads();
    for (int kv = tid; kv < a.K / VEC; kv += 256) {
      bool id = true;
#pragma unroll
      for (int e = 0; e < VEC; ++e) id = id && kmap[kv * VEC + e] == kv * VEC + e;
      kdirect[kv] = id ? 1 : 0;
    }
  }
  __syncthreads();

  // this thread's A rows (input rows of the block) and B rows (weight rows)
  const T* arow[APT];
  const T* crow[APT];                                        // VIRT: cached original row
  const T* drow[APT];                                        // VIRT: compact delta row
#pragma unroll
  for (int j = 0; j < APT; ++j) {
    const int i = tid + j * 256, row = i / KV, kv = i % KV;
    const int xi = m0 + row;
    arow[j] = crow[j] = drow[j] = nullptr;
    if (xi < a.nx) {
      if constexpr (VIRT) {
        crow[j] = reinterpret_cast<const T*>(a.vin.cache) + ((int64_t)a.x0 + xi) * a.K;
        drow[j] = reinterpret_cast<const T*>(a.vin.delta) + ((int64_t)slot * a.nx + xi) * a.vin.HW * a.vin.T;
      } else {
        const int64_t ri = row_index(a.in.mode, (int64_t)slot * a.nx + xi, a.nx, a.x0);
        arow[j] = X + ri * a.K + kv * VEC;
      }
    }
  }
  const T* brow[BPT];
#pragma unroll
  for (int j = 0; j < BPT; ++j) {
    const int i = tid + j * 256;
    brow[j] = nullptr;
    if (i < BN * KV && wrow[i / KV]) brow[j] = wrow[i / KV] + (i % KV) * VEC;
  }

  v4u ra[APT], rb[BPT];
  auto load_chunk = [&](int kc) {
#pragma unroll
    for (int j = 0; j < APT; ++j) {
      const int kv = (tid + j * 256) % KV;
      const int k = kc + kv * VEC;
      v4u v = v4u{0u, 0u, 0u, 0u};
      if constexpr (VIRT) {
        if (crow[j] && k + VEC <= a.K) {
          // the cached original vector, then only the elements the mutant's
          // channel map changes (another cached channel, zero, or a delta entry)
          v = *reinterpret_cast<const v4u*>(crow[j] + k);
          if (!kdirect[k / VEC]) {
            T e8[VEC];
            __builtin_memcpy(e8, &v, 16);
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
              const int code = kmap[k + e];
              if (code != k + e)
                e8[e] = code >= 0 ? crow[j][code] : code != INT_MIN ? drow[j][-1 - code] : T(0);
            }
            __builtin_memcpy(&v, e8, 16);
          }
        } else if (crow[j]) {
          T e8[VEC];
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            T x = T(0);
            if (k + e < a.K) {
              const int code = kmap[k + e];
              if (code >= 0) x = crow[j][code];
              else if (code != INT_MIN) x = drow[j][-1 - code];
            }
            e8[e] = x;
          }
          __builtin_memcpy(&v, e8, 16);
        }
      } else {
        if (arow[j] && k < a.K) v = *reinterpret_cast<const v4u*>(arow[j] + kc);
      }
      ra[j] = v;
    }
#pragma unroll
    for (int j = 0; j < BPT; ++j) {
      const int kv = (tid + j * 256) % KV;
      v4u v = v4u{0u, 0u, 0u, 0u};
      if (brow[j] && kc + kv * VEC < a.K) v = *reinterpret_cast<const v4u*>(brow[j] + kc);
      rb[j] = v;
    }
  };
  auto store_chunk = [&]() {
#pragma unroll
    for (int j = 0; j < APT; ++j) {
      const int i = tid + j * 256;
      *reinterpret_cast<v4u*>(&As[(i / KV) * LD + (i % KV) * VEC]) = ra[j];
    }
#pragma unroll
    for (int j = 0; j < BPT; ++j) {
      const int i = tid + j * 256;
      if (i < BN * KV) *reinterpret_cast<v4u*>(&Bs[(i / KV) * LD + (i % KV) * VEC]) = rb[j];
    }
  };

  // output slot, channel and bias of each of the lane's columns, loaded
  // before the k loop and completed there: left pending into the branchy
  // epilogue, each store would wait for every outstanding memory operation
  const float* __restrict__ bias = a.btab[slot];
  int cslot[TN], cchan[TN];
  float cbias[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int n = n0 + wn * WN + j * 16 + (lane & 15);
    cslot[j] = slot; cchan[j] = n; cbias[j] = 0.f;
    if (n < ncol) {
      if (a.cols) {
        const DeltaCol cd = a.cols[n];
        cslot[j] = a.slot0 + cd.slot - a.col_slot0;
        cchan[j] = a.delta_T > 0 ? cd.t : cd.c;
        cbias[j] = a.btab[cslot[j]][cd.c];
      } else {
        cbias[j] = bias[n];
      }
    }
    asm volatile("" ::"v"(cslot[j]), "v"(cchan[j]), "v"(cbias[j]));
  }

  v4f acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  load_chunk(0);
  for (int kc = 0; kc < a.K; kc += BK) {
    store_chunk();
    __syncthreads();
    if (kc + BK < a.K) load_chunk(kc + BK);                  // next chunk in flight
    if constexpr (sizeof(T) == 4) {
#pragma unroll
      for (int ks = 0; ks < BK / 4; ++ks) {
        float av[TM], bv[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) av[i] = As[(wm * WM + i * 16 + (lane & 15)) * LD + ks * 4 + (lane >> 4)];
#pragma unroll
        for (int j = 0; j < TN; ++j) bv[j] = Bs[(wn * WN + j * 16 + (lane & 15)) * LD + ks * 4 + (lane >> 4)];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], bv[j], acc[i][j], 0, 0, 0);
      }
    } else {
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
    }
    __syncthreads();
  }

  const int orow = a.cols && a.delta_T > 0 ? a.delta_T : a.Cout;   // elements per output row
  // fp32 outputs of whole layers (no gathered columns, no fused kill) with
  // 16-byte aligned rows: each wave stages one 16-column slice of its
  // tile at a time in the (now idle) weight tile and writes it back as
  // 16-byte vectors, a quarter of the store instructions of one element per lane
  constexpr int SST = 20;                                    // floats per staged row
  if constexpr (sizeof(T) == 4 && LSN == 1 && BN * LD >= 4 * WM * SST) {
    if (a.write_out && !a.cols && (a.Cout & 3) == 0 && ((uintptr_t)a.out & 15) == 0) {
      float* const st = reinterpret_cast<float*>(Bs) + wave * WM * SST;
      float* const out = reinterpret_cast<float*>(a.out);
#pragma unroll
      for (int j = 0; j < TN; ++j) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            st[(i * 16 + (lane >> 4) * 4 + e) * SST + (lane & 15)] = act(acc[i][j][e] + cbias[j], a.relu);
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int p = 0; p < WM * 4 / 64; ++p) {
          const int idx = p * 64 + lane, r = idx >> 2, q = idx & 3;
          const v4f v = *reinterpret_cast<const v4f*>(&st[r * SST + q * 4]);
          const int xo = m0 + wm * WM + r;
          const int n = n0 + wn * WN + j * 16 + q * 4;
          if (xo < a.nx && n < a.Cout) {
            const int64_t ro = a.out_mode == MODE_BUF ? (int64_t)slot * a.nx + xo : (int64_t)a.x0 + xo;
            *reinterpret_cast<v4f*>(out + ro * a.Cout + n) = v;
          }
        }
        __builtin_amdgcn_wave_barrier();
      }
      return;
    }
  }
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int nl = wn * WN + j * 16 + (lane & 15);
    const int n = n0 + nl;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int rl = wm * WM + i * 16 + (lane >> 4) * 4 + e;
        float v = acc[i][j][e] + cbias[j];
        v = act(v, a.relu);
        if (a.write_out && n < ncol && m0 + rl < a.nx) {
          // row r = slot * nx + xi of the chunk: buffer row r, or cache row x0 + xi
          const int xo = m0 + rl;
          const int64_t ro = a.out_mode == MODE_BUF ? (int64_t)cslot[j] * a.nx + xo : (int64_t)a.x0 + xo;
          store_out<T>(a.out, a.out_f32, ro * orow + cchan[j], v);
        }
        if constexpr (LSN > 1) {
          if (a.do_kill) Ls[rl * (BN + 1) + nl] = v;
        }
      }
    }
  }
  if constexpr (LSN > 1) {
    if (!a.do_kill) return;
    __syncthreads();
    if (wave != 0) return;
    const int xi = m0 + lane;
    const bool valid = xi < a.nx;
    bool kill = false;
    if (valid) {
      const float* z = &Ls[lane * (BN + 1)];
      float best = -INFINITY;
      int arg = 0, bad = 0;
      for (int c = 0; c < a.Cout; ++c) {
        const float v = z[c];
        if (!isfinite(v)) { ++bad; continue; }
        if (v > best) { best = v; arg = c; }
      }
      if (bad) atomicAdd(a.nonfinite, (unsigned long long)bad);
      const int x = a.x0 + xi;
      kill = a.orig_ok[x] && arg != a.label[x];
      if (a.logits_out)
        for (int c = 0; c < a.Cout; ++c) a.logits_out[(int64_t)x * a.Cout + c] = z[c];
    }
    const unsigned long long word = __ballot(kill);
    if (lane == 0 && a.kill_words && m0 < a.nx)
      a.kill_words[(int64_t)a.slot_mutant[slot] * a.nwords + (a.x0 + m0) / 64] = word;
  }
}

template <typename T, bool VIRT>
static hipError_t dense_dispatch(const DenseArgs& a, dim3 grid, int bn, hipStream_t s) {
  const size_t lds = VIRT ? (size_t)a.K * 4 + (size_t)(a.K + 15) / 16 * 16 : 0;
  switch (bn) {
    case 16: hipLaunchKernelGGL((dense_kernel<T, 16, 4, VIRT, 64>), grid, dim3(256), lds, s, a); break;
    case 32: hipLaunchKernelGGL((dense_kernel<T, 32, 4, VIRT, 64>), grid, dim3(256), lds, s, a); break;
    case 64: hipLaunchKernelGGL((dense_kernel<T, 64, 2, VIRT, 64>), grid, dim3(256), lds, s, a); break;
    case 96: hipLaunchKernelGGL((dense_kernel<T, 96, 2, VIRT, 64>), grid, dim3(256), lds, s, a); break;
    case 128: hipLaunchKernelGGL((dense_kernel<T, 128, 2, VIRT, 64>), grid, dim3(256), lds, s, a); break;
    default: hipLaunchKernelGGL((dense_kernel<T, 256, 1, VIRT, 64>), grid, dim3(256), lds, s, a); break;
  }
  return hipGetLastError();
}

int dense_bn(int cout) {
  return cout <= 16 ? 16 : cout <= 32 ? 32 : cout <= 64 ? 64 : cout <= 96 ? 96 : cout <= 128 ? 128 : 256;
}

hipError_t launch_dense(const DenseArgs& a, int nslots, int dtype, hipStream_t s) {
  if (nslots <= 0 || a.nx <= 0) return hipSuccess;
  if (a.cols && (a.do_kill || a.vin.chmap || a.in.mode != MODE_CACHE || a.ncols <= 0))
    return hipErrorInvalidValue;
  if (a.cols) nslots = 1;
  const int ncol = a.cols ? a.ncols : a.Cout;
  const int bn = dense_bn(ncol);
  const int bm = 64;
  dim3 grid((unsigned)((a.nx + bm - 1) / bm), (unsigned)nslots, (unsigned)((ncol + bn - 1) / bn));
  if (a.do_kill && (grid.z != 1 || bn > 64)) return hipErrorInvalidValue;
  if (a.vin.chmap) {
    if (a.K > 4096) return hipErrorInvalidValue;
    return dtype == 0 ? dense_dispatch<float, true>(a, grid, bn, s) : dense_dispatch<bf16_t, true>(a, grid, bn, s);
  }
  return dtype == 0 ? dense_dispatch<float, false>(a, grid, bn, s) : dense_dispatch<bf16_t, false>(a, grid, bn, s);
}

}  // namespace mure
