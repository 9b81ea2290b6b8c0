// Element-wise layers, the channel-patch (delta) kernel at the first mutated
// layer, the kill reduction, labels, scoring and copy-on-write mutation.
#include "dev.hpp"

namespace mure {

// ---------------------------------------------------------------- ADD
// out = ReLU?(float(a) + float(s')) with s' = s, or for option A
// s'[y][x][c] = s[2y][2x][c - before] inside the copied channel range, else 0.
//
// Vector form: one 16-byte vector (VEC channels of one pixel) per item, with
// multiply-high divisors for the row / pixel / channel-vector decode.  Needs
// C % VEC == 0 and, for option A, a channel offset and C_s that are whole
// vectors (a vector of the shortcut is then wholly inside or outside).
template <typename T>
__global__ __launch_bounds__(256) void add_vec_kernel(AddArgs a, int total_v, DivU32 dper, DivU32 dnx,
                                                      DivU32 dcv, DivU32 dw) {
  constexpr int VEC = 16 / sizeof(T);
  const int64_t per = (int64_t)a.H * a.W * a.C;
  const int before = (a.C - a.Cs) / 2;
  for (int i = (int)(blockIdx.x * 256 + threadIdx.x); i < total_v; i += (int)(gridDim.x * 256)) {
    int r, e, sl, xi;
    divmodu(dper, (uint32_t)i, r, e);                // e = pixel * (C / VEC) + cv
    divmodu(dnx, (uint32_t)r, sl, xi);
    const T* ap = reinterpret_cast<const T*>(a.a.p) + row_at(a.a.mode, sl, xi, a.nx, a.x0) * a.a.row_elems;
    const T* sp = reinterpret_cast<const T*>(a.s.p) + row_at(a.s.mode, sl, xi, a.nx, a.x0) * a.s.row_elems;
    const v4u av = *reinterpret_cast<const v4u*>(ap + (int64_t)e * VEC);
    v4u sv = v4u{0u, 0u, 0u, 0u};
    if (a.shortcut == 0) {
      sv = *reinterpret_cast<const v4u*>(sp + (int64_t)e * VEC);
    } else {
      int pix, cv, y, x;
      divmodu(dcv, (uint32_t)e, pix, cv);
      divmodu(dw, (uint32_t)pix, y, x);
      const int cs = cv * VEC - before;
      if (cs >= 0 && cs < a.Cs) sv = *reinterpret_cast<const v4u*>(sp + ((int64_t)(2 * y) * a.Ws + 2 * x) * a.Cs + cs);
    }
    T x8[VEC], s8[VEC];
    __builtin_memcpy(x8, &av, 16);
    __builtin_memcpy(s8, &sv, 16);
    T* const op = reinterpret_cast<T*>(a.out);
    const int64_t o = row_at(a.out_mode, sl, xi, a.nx, a.x0) * per + (int64_t)e * VEC;
    if (a.out_f32) {
      float* const of = reinterpret_cast<float*>(a.out) + o;
#pragma unroll
      for (int j = 0; j < VEC; ++j) of[j] = act(to_f<T>(x8[j]) + to_f<T>(s8[j]), a.relu);
    } else {
      T o8[VEC];
#pragma unroll
      for (int j = 0; j < VEC; ++j) o8[j] = from_f<T>(act(to_f<T>(x8[j]) + to_f<T>(s8[j]), a.relu));
      v4u ov;
      __builtin_memcpy(&ov, o8, 16);
      *reinterpret_cast<v4u*>(op + o) = ov;
    }
  }
}

template <typename T>
__global__ void add_kernel(AddArgs a) {
  const int64_t per = (int64_t)a.H * a.W * a.C;
  const int64_t total = a.rows * per;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / per;
    const int64_t e = i % per;
    const int c = (int)(e % a.C);
    const int64_t pix = e / a.C;
    const T* ap = reinterpret_cast<const T*>(a.a.p) + row_index(a.a.mode, r, a.nx, a.x0) * a.a.row_elems;
    const T* sp = reinterpret_cast<const T*>(a.s.p) + row_index(a.s.mode, r, a.nx, a.x0) * a.s.row_elems;
    float sv;
    if (a.shortcut == 0) {
      sv = to_f<T>(sp[e]);
    } else {
      const int y = (int)(pix / a.W), x = (int)(pix % a.W);
      const int cs = c - (a.C - a.Cs) / 2;
      sv = (cs >= 0 && cs < a.Cs) ? to_f<T>(sp[((int64_t)(2 * y) * a.Ws + 2 * x) * a.Cs + cs]) : 0.f;
    }
    float v = to_f<T>(ap[e]) + sv;
    v = act(v, a.relu);
    store_out<T>(a.out, a.out_f32, row_index(a.out_mode, r, a.nx, a.x0) * per + e, v);
  }
}

// ---------------------------------------------------------------- GAP
// sum over the H*W pixels in order (float32), times 1/(H*W), then rounding.
template <typename T>
__global__ void gap_kernel(GapArgs a) {
  const int64_t total = a.rows * a.C;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / a.C;
    const int c = (int)(i % a.C);
    const T* ip = reinterpret_cast<const T*>(a.in.p) + row_index(a.in.mode, r, a.nx, a.x0) * a.in.row_elems;
    // eight loads in flight, then their sums in pixel order
    float s = 0.f;
    int p = 0;
    for (; p + 8 <= a.P; p += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = to_f<T>(ip[(int64_t)(p + u) * a.C + c]);
#pragma unroll
      for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; p < a.P; ++p) s += to_f<T>(ip[(int64_t)p * a.C + c]);
    store_out<T>(a.out, a.out_f32, row_index(a.out_mode, r, a.nx, a.x0) * a.C + c, s * (1.0f / (float)a.P));
  }
}

// ---------------------------------------------------------------- channel patch
// Node mmi of an effect-block / switch mutant: the original's output with
// channel c taken from original channel chmap[c] (-1: zero).  Bitwise copy.
// A block copies `rows` consecutive inputs of one slot: a contiguous span of
// the cache and of the chunk buffer.  The span goes through LDS in tiles of
// whole pixels (one coalesced 16-byte load per vector); 16-byte vectors
// whose channels the map keeps in place are copied whole, the others
// gathered element by element from the staged pixel (gathered from global
// memory, two bytes a load, they had cost most of the kernel's time).
constexpr int PATCH_MAXC = 4096;
constexpr int PATCH_TILE_B = 32768;                     // staged bytes per tile

template <typename E>
__global__ __launch_bounds__(256) void patch_kernel(PatchArgs a, int rows, DivU32 dcv, DivU32 dc) {
  constexpr int VEC = 16 / sizeof(E);
  constexpr int TV_MAX = PATCH_TILE_B / 16;             // vectors per tile, at most
  __shared__ int map[PATCH_MAXC];
  __shared__ unsigned char keep[PATCH_MAXC / VEC];
  __shared__ __attribute__((aligned(16))) v4u tile[TV_MAX];
  const int tid = threadIdx.x;
  const int sl = (int)blockIdx.y;
  const int32_t* cm = a.chmap + (int64_t)(a.chmap_slot0 + sl) * a.C;
  for (int c = tid; c < a.C; c += 256) map[c] = cm[c];
  __syncthreads();
  const bool vec = a.C % VEC == 0;
  const int CV = a.C / VEC;
  if (vec) {
    for (int v = tid; v < CV; v += 256) {
      bool k = true;
#pragma unroll
      for (int j = 0; j < VEC; ++j) k = k && map[v * VEC + j] == v * VEC + j;
      keep[v] = k ? 1 : 0;
    }
    __syncthreads();
  }
  const int xi0 = (int)blockIdx.x * rows;
  const int nr = min(rows, a.nx - xi0);
  if (nr <= 0) return;
  const int per = a.P * a.C;
  const E* src = reinterpret_cast<const E*>(a.cache) + ((int64_t)a.x0 + xi0) * per;
  E* dst = reinterpret_cast<E*>(a.out) + ((int64_t)(a.slot0 + sl) * a.nx + xi0) * per;
  if (vec && CV <= TV_MAX) {
    constexpr int PB = TV_MAX / 256;                    // vectors per thread and tile
    const int TV = TV_MAX / CV * CV;                    // a tile holds whole pixels
    const int nv = nr * (per / VEC);
    const E* const te = reinterpret_cast<const E*>(tile);
    for (int t0 = 0; t0 < nv; t0 += TV) {
      const int tn = min(TV, nv - t0);
      // the tile's cached vectors, all loads first
      v4u ld[PB];
#pragma unroll
      for (int u = 0; u < PB; ++u) {
        const int v = tid + 256 * u;
        if (v < tn) ld[u] = reinterpret_cast<const v4u*>(src)[t0 + v];
      }
#pragma unroll
      for (int u = 0; u < PB; ++u) {
        const int v = tid + 256 * u;
        if (v < tn) tile[v] = ld[u];
      }
      __syncthreads();
#pragma unroll
      for (int u = 0; u < PB; ++u) {
        const int v = tid + 256 * u;
        if (v >= tn) continue;
        const int cv = (int)((uint32_t)v - divu(dcv, (uint32_t)v) * (uint32_t)CV);
        v4u o;
        if (keep[cv]) {
          o = tile[v];
        } else {
          const int pix0 = (v - cv) * VEC;              // the pixel's first element in the tile
          E t[VEC];
#pragma unroll
          for (int j = 0; j < VEC; ++j) {
            const int m = map[cv * VEC + j];
            t[j] = m < 0 ? E(0) : te[pix0 + m];
          }
          __builtin_memcpy(&o, t, 16);
        }
        reinterpret_cast<v4u*>(dst)[t0 + v] = o;
      }
      __syncthreads();                                  // the tile is read before the next one lands
    }
  } else {
    const int ne = nr * per;
    for (int e = tid; e < ne; e += 256) {
      const int c = (int)(e - divu(dc, (uint32_t)e) * a.C);
      const int m = map[c];
      dst[e] = m < 0 ? E(0) : src[e - c + m];
    }
  }
}

// ---------------------------------------------------------------- kill reduction
// One thread per (slot, input); a wavefront covers 64 consecutive inputs of
// one slot, i.e. exactly one 64-bit kill word (x0 is a multiple of 64).
__global__ __launch_bounds__(256) void kill_kernel(KillArgs a) {
  const int sl = a.slot0 + (int)blockIdx.y;
  const int xi = (int)blockIdx.x * 256 + (int)threadIdx.x;
  const bool valid = xi < a.nx;
  bool kill = false;
  if (valid) {
    const float* z = a.logits + ((int64_t)sl * a.nx + xi) * a.C;
    float best = z[0];
    int arg = 0, bad = !isfinite(best);
    if (bad) best = -INFINITY;
    for (int c = 1; c < a.C; ++c) {
      const float v = z[c];
      if (!isfinite(v)) { ++bad; continue; }
      if (v > best) { best = v; arg = c; }
    }
    if (bad) atomicAdd(a.nonfinite, (unsigned long long)bad);
    const int x = a.x0 + xi;
    kill = a.orig_ok[x] && arg != a.label[x];
    if (a.logits_out)
      for (int c = 0; c < a.C; ++c) a.logits_out[(int64_t)x * a.C + c] = z[c];
  }
  const unsigned long long word = __ballot(kill);
  const int wave_first = (int)blockIdx.x * 256 + ((int)threadIdx.x & ~63);
  if ((threadIdx.x & 63) == 0 && wave_first < a.nx && a.kill_words) {
    const int64_t m = a.slot_mutant[sl];
    a.kill_words[m * a.nwords + (a.x0 + wave_first) / 64] = word;
  }
}

// ---------------------------------------------------------------- labels
__global__ void labels_kernel(LabelArgs a) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= a.N) return;
  const float* z = a.logits + x * a.C;
  float best = -INFINITY;
  int arg = 0, bad = 0;
  for (int c = 0; c < a.C; ++c) {
    const float v = z[c];
    if (!isfinite(v)) { ++bad; continue; }
    if (v > best) { best = v; arg = c; }
  }
  if (bad) atomicAdd(a.nonfinite, (unsigned long long)bad);
  const int lab = a.given ? a.given[x] : arg;
  a.label[x] = lab;
  a.ok[x] = (uint8_t)(arg == lab);
  atomicOr(&a.class_mask[lab >> 6], 1ull << (lab & 63));
}

// ---------------------------------------------------------------- score
// Per mutant: kills = popcount of its words; killingLabels mask = OR of
// 1 << label(x) over killed x.  Integer only: order-independent.
__global__ __launch_bounds__(256) void score_kernel(ScoreArgs a) {
  __shared__ unsigned long long mask[8];
  __shared__ unsigned long long count;
  const int64_t m = blockIdx.x;
  if (threadIdx.x < 8) mask[threadIdx.x] = 0;
  if (threadIdx.x == 0) count = 0;
  __syncthreads();
  unsigned long long cnt = 0;
  for (int64_t w = threadIdx.x; w < a.nwords; w += blockDim.x) {
    unsigned long long bits = a.kill_words[m * a.nwords + w];
    cnt += __popcll(bits);
    while (bits) {
      const int b = __ffsll((long long)bits) - 1;
      bits &= bits - 1;
      const int lab = a.label[w * 64 + b];
      atomicOr(&mask[lab >> 6], 1ull << (lab & 63));
    }
  }
  atomicAdd(&count, cnt);
  __syncthreads();
  if (threadIdx.x == 0) a.kills[m] = (int64_t)count;
  if ((int)threadIdx.x < a.mask_words) a.masks[m * a.mask_words + threadIdx.x] = mask[threadIdx.x];
}

// ---------------------------------------------------------------- copy-on-write mutation
// One block per (mutant, layer) copy: copy the original parameters, then
// apply that mutant's records on this layer in order.  Weight (neuron n, k)
// is element n rs + k ks of the layer's array, or for chunk-major halo
// weights halo_w_index(n, k / C_in, k % C_in, C_out).
template <typename T>
__global__ __launch_bounds__(256) void cow_kernel(const CowArgs* args, const DevRecord* recs,
                                                  const float* noise) {
  const CowArgs c = args[blockIdx.x];
  const T* ws = reinterpret_cast<const T*>(c.w_src);
  T* wd = reinterpret_cast<T*>(c.w_dst);
  const int64_t n = (int64_t)c.c_out * c.fan_in;
  // the copy in 16-byte vectors when both arrays allow it (the pool's
  // copies are 256-byte aligned; the originals are device allocations)
  const int64_t nb = n * (int64_t)sizeof(T);
  if (nb % 16 == 0 && ((uintptr_t)ws | (uintptr_t)wd) % 16 == 0) {
    const v4u* vs = reinterpret_cast<const v4u*>(ws);
    v4u* vd = reinterpret_cast<v4u*>(wd);
    for (int64_t i = threadIdx.x; i < nb / 16; i += blockDim.x) vd[i] = vs[i];
  } else {
    for (int64_t i = threadIdx.x; i < n; i += blockDim.x) wd[i] = ws[i];
  }
  for (int i = threadIdx.x; i < c.c_out; i += blockDim.x) c.b_dst[i] = c.b_src[i];
  __syncthreads();
  // element k (k = tap C_in + ci for a convolution) of neuron nr's weights
  auto at = [&](int nr, int64_t k) -> T& {
    if (c.halo_c > 0) return wd[halo_w_index(nr, (int)(k / c.halo_c), (int)(k % c.halo_c), c.c_out)];
    return wd[(int64_t)nr * c.rs + k * c.ks];
  };
  for (int ri = c.rec0; ri < c.rec1; ++ri) {
    const DevRecord r = recs[ri];
    if (r.op == 0) {                      // Gaussian fuzz: float32 add, then round
      const float* eps = noise + r.noise_off;
      for (int64_t k = threadIdx.x; k < c.fan_in; k += blockDim.x) {
        T& w = at(r.neuron, k);
        w = from_f<T>(to_f<T>(w) + eps[k]);
      }
    } else if (r.op == 1) {               // effect block
      for (int64_t k = threadIdx.x; k < c.fan_in; k += blockDim.x) at(r.neuron, k) = T(0);
      if (threadIdx.x == 0) c.b_dst[r.neuron] = 0.f;
    } else if (r.op == 2) {               // activation inverse (exact sign flip)
      for (int64_t k = threadIdx.x; k < c.fan_in; k += blockDim.x) {
        T& w = at(r.neuron, k);
        if constexpr (sizeof(T) == 2) w = (T)(w ^ 0x8000u);
        else w = -w;
      }
      if (threadIdx.x == 0) c.b_dst[r.neuron] = -c.b_dst[r.neuron];
    } else if (r.op == 4) {               // weight shuffle: row[k] <- old row[perm[k]]
      float* scratch = const_cast<float*>(noise) + r.scratch_off;
      const int32_t* perm = reinterpret_cast<const int32_t*>(noise + r.noise_off);
      for (int64_t k = threadIdx.x; k < c.fan_in; k += blockDim.x) scratch[k] = to_f<T>(at(r.neuron, k));
      __syncthreads();
      for (int64_t k = threadIdx.x; k < c.fan_in; k += blockDim.x) at(r.neuron, k) = from_f<T>(scratch[perm[k]]);
    } else {                              // neuron switch
      for (int64_t k = threadIdx.x; k < c.fan_in; k += blockDim.x) {
        T& u = at(r.neuron, k);
        T& v = at(r.partner, k);
        const T t = u; u = v; v = t;
      }
      if (threadIdx.x == 0) {
        const float t = c.b_dst[r.neuron]; c.b_dst[r.neuron] = c.b_dst[r.partner]; c.b_dst[r.partner] = t;
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------- changed channel groups
// A block stages a tile of GP_TILE pixel rows of the cache in LDS (one
// coalesced read of each row), then writes the tile's 16-byte group vector of
// every entry (slot, group): consecutive lanes take consecutive pixels of one
// entry, so the side plane is written in whole runs.  A channel the entry
// takes from another channel of the row (a switch) is read from the tile; one
// it zeroes or recomputes comes from 0 or the compact delta rows.  The
// entries' maps are staged in LDS (at most GROUP_PATCH_MAXE per launch).
constexpr int GROUP_PATCH_MAXE = 256;
constexpr int GP_TILE_BYTES = 32768;                   // cached bytes per tile
constexpr int GP_TILE_PAD = 16;                         // per row: spreads the rows over the banks
__global__ __launch_bounds__(256) void group_patch_kernel(GroupPatchArgs a, int px_tile) {
  __shared__ int smap[GROUP_PATCH_MAXE][8];
  __shared__ int sgrp[GROUP_PATCH_MAXE], sslot[GROUP_PATCH_MAXE];
  __shared__ __attribute__((aligned(16))) unsigned char tile[GP_TILE_BYTES + 256 * GP_TILE_PAD];
  for (int t = threadIdx.x; t < a.n_ent * 8; t += 256) {
    const int e = t >> 3, j = t & 7;
    const int slot = a.ent[2 * e], g = a.ent[2 * e + 1];
    smap[e][j] = a.chmap[(int64_t)slot * a.C + 8 * g + j];
    if (j == 0) { sgrp[e] = g; sslot[e] = slot; }
  }
  const int G = a.C / 8, RS = a.C * 2 + GP_TILE_PAD;   // row stride in the tile, bytes
  const int64_t npx = (int64_t)a.nx * a.P;
  const uint16_t* __restrict__ cache = reinterpret_cast<const uint16_t*>(a.cache);
  const uint16_t* __restrict__ delta = reinterpret_cast<const uint16_t*>(a.delta);
  v4u* side = reinterpret_cast<v4u*>(a.side);
  for (int64_t i0 = (int64_t)blockIdx.x * px_tile; i0 < npx; i0 += (int64_t)gridDim.x * px_tile) {
    const int npt = npx - i0 < px_tile ? (int)(npx - i0) : px_tile;
    __syncthreads();                                    // the previous tile is consumed (and smap is staged)
    for (int t = threadIdx.x; t < npt * G; t += 256) {
      const int p = t / G, g = t % G;
      *reinterpret_cast<v4u*>(tile + p * RS + g * 16) =
          *reinterpret_cast<const v4u*>(cache + (i0 + p) * a.C + 8 * g);
    }
    __syncthreads();
    for (int t = threadIdx.x; t < a.n_ent * npt; t += 256) {
      const int e = t / npt, p = t % npt;
      const int g = sgrp[e];
      const uint16_t* row = reinterpret_cast<const uint16_t*>(tile + p * RS);
      v4u v = *reinterpret_cast<const v4u*>(row + 8 * g);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int m = smap[e][j];
        if (m == 8 * g + j) continue;
        const uint32_t x = m >= 0 ? row[m]
                         : m == -1 ? 0u : delta[((int64_t)(sslot[e] - a.slot0) * npx + i0 + p) * a.T + (-2 - m)];
        v[j >> 1] = (v[j >> 1] & (0xffff0000u >> (16 * (j & 1)))) | (x << (16 * (j & 1)));
      }
      side[(int64_t)e * npx + i0 + p] = v;
    }
  }
}

// ---------------------------------------------------------------- row copy (FLATTEN)
template <typename E>
__global__ void copy_rows_kernel(TensorArg src, E* dst, int64_t rows, int nx, int x0) {
  const int64_t total = rows * src.row_elems;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / src.row_elems, e = i % src.row_elems;
    dst[i] = reinterpret_cast<const E*>(src.p)[row_index(src.mode, r, nx, x0) * src.row_elems + e];
  }
}

// ---------------------------------------------------------------- launchers
static unsigned grid_for(int64_t total, int block = 256) {
  int64_t g = (total + block - 1) / block;
  if (g > 65536LL * 8) g = 65536LL * 8;
  return (unsigned)(g < 1 ? 1 : g);
}

hipError_t launch_add(const AddArgs& a, int dtype, hipStream_t s) {
  const int64_t total = a.rows * a.H * a.W * a.C;
  if (total == 0) return hipSuccess;
  const int vec = dtype == 0 ? 4 : 8;
  const int64_t per_v = (int64_t)a.H * a.W * a.C / vec;
  const bool vec_ok = a.C % vec == 0 && total / vec < (1 << 30) && a.rows < (1 << 30) && a.a.row_elems % vec == 0 &&
                      a.s.row_elems % vec == 0 &&
                      (a.shortcut == 0 || (((a.C - a.Cs) / 2) % vec == 0 && a.Cs % vec == 0));
  if (vec_ok) {
    const int total_v = (int)(total / vec);
    const DivU32 dper = make_divu32((uint32_t)per_v), dnx = make_divu32((uint32_t)std::max(1, a.nx));
    const DivU32 dcv = make_divu32((uint32_t)(a.C / vec)), dw = make_divu32((uint32_t)std::max(1, a.W));
    if (dtype == 0)
      hipLaunchKernelGGL(add_vec_kernel<float>, dim3(grid_for(total_v)), dim3(256), 0, s, a, total_v, dper, dnx, dcv, dw);
    else
      hipLaunchKernelGGL(add_vec_kernel<bf16_t>, dim3(grid_for(total_v)), dim3(256), 0, s, a, total_v, dper, dnx, dcv, dw);
    return hipGetLastError();
  }
  if (dtype == 0) hipLaunchKernelGGL(add_kernel<float>, dim3(grid_for(total)), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(add_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gap(const GapArgs& a, int dtype, hipStream_t s) {
  const int64_t total = a.rows * a.C;
  if (total == 0) return hipSuccess;
  if (dtype == 0) hipLaunchKernelGGL(gap_kernel<float>, dim3(grid_for(total)), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(gap_kernel<bf16_t>, dim3(grid_for(total)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_patch(const PatchArgs& a, hipStream_t s) {
  if (a.nslots <= 0 || a.nx <= 0 || a.P <= 0 || a.C <= 0) return hipSuccess;
  if (a.C > PATCH_MAXC || a.nslots > 65535 || (a.esize != 2 && a.esize != 4)) return hipErrorInvalidValue;
  const int64_t per = (int64_t)a.P * a.C;
  // about 16K elements per block
  const int rows = (int)std::max<int64_t>(1, std::min<int64_t>(a.nx, 16384 / per));
  if (per * rows >= INT32_MAX) return hipErrorInvalidValue;
  const int vec = 16 / a.esize;
  const DivU32 dcv = make_divu32((uint32_t)std::max(1, a.C / vec)), dc = make_divu32((uint32_t)a.C);
  dim3 grid((unsigned)((a.nx + rows - 1) / rows), (unsigned)a.nslots);
  if (a.esize == 4) hipLaunchKernelGGL(patch_kernel<uint32_t>, grid, dim3(256), 0, s, a, rows, dcv, dc);
  else hipLaunchKernelGGL(patch_kernel<uint16_t>, grid, dim3(256), 0, s, a, rows, dcv, dc);
  return hipGetLastError();
}

hipError_t launch_kill(const KillArgs& a, hipStream_t s) {
  if (a.nslots <= 0 || a.nx <= 0) return hipSuccess;
  dim3 grid((unsigned)((a.nx + 255) / 256), (unsigned)a.nslots);
  hipLaunchKernelGGL(kill_kernel, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_labels(const LabelArgs& a, hipStream_t s) {
  if (a.N == 0) return hipSuccess;
  hipLaunchKernelGGL(labels_kernel, dim3((unsigned)((a.N + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_score(const ScoreArgs& a, int n_mutants, hipStream_t s) {
  if (n_mutants == 0) return hipSuccess;
  hipLaunchKernelGGL(score_kernel, dim3((unsigned)n_mutants), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_group_patch(const GroupPatchArgs& a0, hipStream_t s) {
  if (a0.n_ent <= 0 || a0.nx <= 0) return hipSuccess;
  if (a0.C % 8 || a0.C * 2 > GP_TILE_BYTES || a0.P <= 0) return hipErrorInvalidValue;
  const int64_t npx = (int64_t)a0.nx * a0.P;
  // pixels per tile: the cache rows that fit GP_TILE_BYTES, at most 256
  const int px_tile = std::min(256, GP_TILE_BYTES / (a0.C * 2));
  const unsigned gx = (unsigned)std::min<int64_t>((npx + px_tile - 1) / px_tile, 4096);
  // entries in pieces that fit the kernel's LDS table
  for (int e0 = 0; e0 < a0.n_ent; e0 += GROUP_PATCH_MAXE) {
    GroupPatchArgs a = a0;
    a.n_ent = std::min(GROUP_PATCH_MAXE, a0.n_ent - e0);
    a.ent = a0.ent + 2 * e0;
    a.side = reinterpret_cast<v4u*>(a0.side) + (int64_t)e0 * npx;
    hipLaunchKernelGGL(group_patch_kernel, dim3(gx), dim3(256), 0, s, a, px_tile);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_cow(const CowArgs* d_args, int n_copies, const DevRecord* d_recs,
                      const float* d_noise, int dtype, hipStream_t s) {
  if (n_copies == 0) return hipSuccess;
  if (dtype == 0)
    hipLaunchKernelGGL(cow_kernel<float>, dim3((unsigned)n_copies), dim3(256), 0, s, d_args, d_recs, d_noise);
  else
    hipLaunchKernelGGL(cow_kernel<bf16_t>, dim3((unsigned)n_copies), dim3(256), 0, s, d_args, d_recs, d_noise);
  return hipGetLastError();
}

hipError_t launch_copy_rows(const TensorArg& src, void* dst, int64_t rows, int nx, int x0,
                            int esize, hipStream_t s) {
  const int64_t total = rows * src.row_elems;
  if (total == 0) return hipSuccess;
  if (esize == 4)
    hipLaunchKernelGGL(copy_rows_kernel<uint32_t>, dim3(grid_for(total)), dim3(256), 0, s, src,
                       reinterpret_cast<uint32_t*>(dst), rows, nx, x0);
  else
    hipLaunchKernelGGL(copy_rows_kernel<uint16_t>, dim3(grid_for(total)), dim3(256), 0, s, src,
                       reinterpret_cast<uint16_t*>(dst), rows, nx, x0);
  return hipGetLastError();
}

// ---------------------------------------------------------------- zero fill
__global__ __launch_bounds__(256) void zero_u64_kernel(uint64_t* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) p[i] = 0;
}

hipError_t launch_zero_u64(uint64_t* p, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(zero_u64_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

}  // namespace mure
