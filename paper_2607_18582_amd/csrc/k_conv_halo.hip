// bf16 3x3 convolutions with stride 1 and padding 1 (C_in % 16 == 0, square
// images of width 8, 16, 32 or 64) as an implicit GEMM on MFMA
// (v_mfma_f32_32x32x16_bf16) whose operands both come from LDS.
//
// Tile: 512 output pixels x BN = 32 TN output channels, four waves of 128
// pixels x BN channels (4 x TN accumulator tiles of 32 x 32), two blocks per
// CU (one wave per SIMD each).  The pixels are TR = 512 / W consecutive image
// rows -- a band of one image, or 512 / (H W) whole images -- so a tile never
// mixes two images' borders.
//
// The input channels go in chunks of 16.  Per chunk the block stages in LDS
// (a) the band's input rows plus the row above and below each packed image's
// rows (the halo, zero outside the image), W pixels a row, in blocks of 32
// pixels with the two 8-channel halves of each block side by side,
// [block][half][32][8]: every input element crosses the memory pipeline once
// per block and chunk instead of once per tap as an im2col gather would; and
// (b) the chunk's weights for the tile's columns, [tap][half][column][8].
// One MFMA k-step of 16 is one tap of the chunk, so a chunk is nine k-steps,
// and the A fragment of a tap is the lane's halo entry of the pixel shifted
// by (dy, dx).  A tap that would read column -1 or W reads a zero block
// instead (a per-lane select), so the halo has no border columns.  Both
// fragments of a k-step are 32 consecutive pixels or columns per half wave,
// which ds_read_b128 serves without bank conflicts.  Within a chunk the
// fragments of tap t + 1 are read before the MFMAs of tap t are issued.
//
// The stages are fetched with direct global-to-LDS loads (16 bytes per lane,
// landing at consecutive LDS addresses per instruction), so staging takes no
// registers.  A load instruction fetches one halo block -- the two lanes of
// a pixel read the chunk's 32 bytes of one cache line -- or 1 KB of weights,
// contiguous in the chunk-major weight layout (halo_w_index): an address
// unit that serves about one cache line per two clocks then moves 32 or 128
// bytes per line instead of 16.  The stages are double-buffered: the loads
// of chunk c + 1 are issued before the MFMAs of chunk c and waited for after
// them, one barrier per chunk.
//
// One tile per block.  The epilogue (bias, activation, bf16 rounding) stages
// the tile in LDS and stores whole output rows as 16-byte vectors, with a
// fused ADD (identity or option-A shortcut) or a fused 2x2 max-pool, or the
// gathered delta columns.
//
// Reduction order: k = (chunk of 16 channels, tap, channel), fixed for a node
// shape; every launch of a node (full rows or gathered delta columns) uses it.
#include "dev.hpp"
#include "plan.hpp"

namespace mure {

namespace {
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;

// Compile-time geometry of an instance (image width W, TN column tiles).
template <int W, int TN>
struct HaloGeo {
  static constexpr int NT = 256, BM = 512, TR = BM / W, BN = 32 * TN;
  static constexpr int NPX = conv_halo_cap(W);          // halo pixels a stage holds
  static_assert(NPX % 32 == 0, "the halo is stored in blocks of 32 pixels");
  static constexpr int NQ_HALO = NPX / 32;              // halo load instructions: a block of 32 pixels each
  static constexpr int HZERO = NQ_HALO * 1024;          // a zero block: [half][32][8]
  static constexpr int HALO_B = HZERO + 1024;
  static constexpr int B_B = 9 * 2 * BN * 16;           // weights: [tap][half][column][8]
  static constexpr int STAGE = HALO_B + B_B;
  static constexpr int NQ = NQ_HALO + 9 * 2 * BN / 64;  // load instructions per chunk
  static constexpr int QPW = (NQ + 3) / 4;              // ... per wave
  static constexpr int OLD = BN + 8;                    // staged output row (bf16)
  static constexpr int VPR = BN / 8;                    // 16-byte vectors per output row
};

struct HaloTile {
  int slot, n0, xi0, y0;
};

// Tile t -> (slot, band, column block).  Consecutive tiles go round-robin to
// the 8 XCDs (block b runs on XCD b % 8); on one XCD the column blocks of a
// band take consecutive turns and share its L2 copy of the band's input.
// When bands are parts of one image (H > TR) each XCD takes a contiguous run
// of a slot's bands, so that the blocks running together on it share the
// rows above and below their bands in its L2 (width 64 on resnet18w: 5.85 ->
// 5.39 ms per launch); bands of whole images go round-robin.  When every slot
// reads the same input or shortcut (a prefix-cache tensor, or the cached
// groups of a channel-group read), the slots of a (band, column block) take
// consecutive turns instead of the slots coming one after another, so that
// the band is fetched once per XCD (slot after slot, a cached shortcut was
// streamed from HBM once per slot: 13 GB instead of 7.8 per width-64
// launch).  false: t is padding of that order.
template <int W, int TN>
__device__ __forceinline__ bool halo_decode(const ConvArgs& a, int t, HaloTile& tl) {
  using G = HaloGeo<W, TN>;
  const int bgroups = (a.bands + 7) / 8;
  const int xcd = t & 7, turn = t >> 3, per_slot = bgroups * a.zblocks;
  const bool slot_inner = a.in.mode == MODE_CACHE || a.gin.cache != nullptr || a.gskip.cache != nullptr;
  const int si = slot_inner ? turn % a.halo_slots : turn / per_slot;
  const int rem = slot_inner ? turn / a.halo_slots : turn % per_slot;
  const int bi = rem / a.zblocks;
  const int band = a.H > G::TR ? xcd * bgroups + bi : bi * 8 + xcd;
  if (band >= a.bands) return false;
  tl.slot = a.slot0 + si;
  tl.n0 = (rem % a.zblocks) * G::BN;
  const int64_t r0 = (int64_t)band * G::TR;             // first row of the flattened (input, row) axis
  tl.xi0 = (int)(r0 / a.H);
  tl.y0 = (int)(r0 % a.H);
  return true;
}

// The lane's sources for this wave's load instructions q = wave + 4 s of a
// tile.  q < NQ_HALO fills halo block q: pixels 32 q + (lane & 31), channel
// half lane >> 5, so the two lanes of a pixel read the chunk's 32 bytes from
// one cache line; hs.h[s] is the element offset of that pixel's half from
// the tile's input base hs.in0 at chunk 0 (-1: zeros), or with VIN (input
// read in channel groups) the pixel's index in the launch's rows (the
// group's base comes per chunk).  The other instructions fill 64 consecutive
// [tap][half][column] weight entries, contiguous in the chunk-major weight
// layout; a lane reads the same column, output channel n of its slot's
// weights, in every one of them, from hs.w (nullptr: zeros) plus a
// per-instruction offset.
template <int W, int TN>
struct HaloSrc {
  static constexpr int NH = (HaloGeo<W, TN>::NQ_HALO + 3) / 4;   // halo instructions per wave, at most
  const bf16_t* in0;
  int h[NH];
  const bf16_t* w;
};

template <int W, int TN, bool VIN>
__device__ __forceinline__ void halo_sources(const ConvArgs& a, const HaloTile& tl, int RI, int npx, int wave,
                                             int lane, HaloSrc<W, TN>& hs) {
  using G = HaloGeo<W, TN>;
  const int ncol = a.cols ? a.ncols : a.Cout;
  hs.in0 = reinterpret_cast<const bf16_t*>(a.in.p) +
           row_at(a.in.mode, tl.slot, tl.xi0 < a.nx ? tl.xi0 : 0, a.nx, a.x0) *
               a.in.row_elems;
#pragma unroll
  for (int s = 0; s < HaloSrc<W, TN>::NH; ++s) {
    const int q = wave + 4 * s;
    const int hh = lane >> 5, px = q * 32 + (lane & 31);
    const int im = px / ((RI + 2) * W), rem = px % ((RI + 2) * W);
    const int y = tl.y0 + rem / W - 1, x = rem % W;
    hs.h[s] = -1;
    if (q < G::NQ_HALO && px < npx && tl.xi0 + im < a.nx && (unsigned)y < (unsigned)a.H)
      hs.h[s] = VIN ? (tl.xi0 + im) * a.H * W + y * W + x
                    : (int)(im * a.in.row_elems) + (y * W + x) * a.C + hh * 8;
  }
  // weights: column n0 + lane % BN of the tile; with BN = 32 the upper half
  // wave reads the second channel half of each tap
  const int nc = tl.n0 + lane % G::BN;
  hs.w = nullptr;
  if (nc < ncol) {
    const void* w;
    int n;
    if (a.cols) {
      const DeltaCol cd = a.cols[nc];
      w = a.wtab[a.slot0 + cd.slot - a.col_slot0];
      n = cd.c;
    } else {
      w = a.wtab[tl.slot];
      n = nc;
    }
    hs.w = reinterpret_cast<const bf16_t*>(w) + halo_w_index(n, 0, G::BN == 32 ? 8 * (lane >> 5) : 0, a.Cout);
  }
}

// The chunk at channel c0 of a VIN input: per channel half, the base of its
// 8-channel group (the cache or the group's side plane) and the pixel stride.
__device__ __forceinline__ void halo_group_bases(const GroupIn& gi, int slot, int nx, int c0,
                                                 const bf16_t* (&gb)[2], int (&gst)[2]) {
  const int64_t plane = (int64_t)nx * gi.P * 8;
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const int g = c0 / 8 + hh;
    const int e = gi.src[slot * (gi.C / 8) + g];
    if (e < 0) {
      gb[hh] = reinterpret_cast<const bf16_t*>(gi.cache) + 8 * g;
      gst[hh] = gi.C;
    } else {
      gb[hh] = reinterpret_cast<const bf16_t*>(gi.side) + (int64_t)(e - gi.g0) * plane;
      gst[hh] = 8;
    }
  }
}

// Issue the loads of the chunk at channel c0 (weight entries wc on from
// chunk 0's) into the stage at st.  Lanes past the halo load nothing.
template <int W, int TN, bool VIN>
__device__ __forceinline__ void halo_fetch(unsigned char* st, const HaloSrc<W, TN>& hs, int npx, int wave, int lane,
                                           int c0, int wc, int Cout, const bf16_t* zp,
                                           const bf16_t* const (&gb)[2], const int (&gst)[2]) {
  using G = HaloGeo<W, TN>;
#pragma unroll
  for (int s = 0; s < G::QPW; ++s) {
    const int q = wave + 4 * s;
    if (q >= G::NQ) continue;
    if (q < G::NQ_HALO) {
      if (q * 32 + (lane & 31) < npx) {
        const int e = hs.h[s < HaloSrc<W, TN>::NH ? s : 0];
        const bf16_t* p;
        if constexpr (VIN) {
          const int hh = lane >> 5;
          p = e < 0 ? zp : gb[hh] + (int64_t)e * gst[hh];
        } else {
          p = e < 0 ? zp : hs.in0 + e + c0;
        }
        __builtin_amdgcn_global_load_lds((const void*)p, (lds_void*)(st + q * 1024), 16, 0, 0);
      }
    } else {
      // entries e = 64 (q - NQ_HALO) + lane: tap e / 2BN, half (e / BN) & 1
      const int e0 = (q - G::NQ_HALO) * 64;
      const int tap = e0 / (2 * G::BN), hu = G::BN == 64 ? (e0 / 64) & 1 : 0;
      const bf16_t* p = hs.w ? hs.w + (int64_t)(tap * 2 + hu) * Cout * 8 + wc : zp;
      __builtin_amdgcn_global_load_lds((const void*)p, (lds_void*)(st + G::HALO_B + (q - G::NQ_HALO) * 1024), 16,
                                       0, 0);
    }
  }
}

// Byte offset in a stage of halo pixel p, channel half h: the halo is
// stored in blocks of 32 pixels, [block][half][32][8].
__device__ __forceinline__ int halo_addr(int p, int h) { return (p >> 5) * 1024 + h * 512 + (p & 31) * 16; }

// Fragment bases: lane row (lane & 31) of M tile i is band pixel m, its 8 k
// are channels 8 h of the chunk (h = lane >> 5).  The tap (dy, dx) reads halo
// pixel hp + (dy + 1) W + dx, where hp is the pixel's column in the halo row
// above it.  A.r[i] is the entry of hp; for W >= 32 the rows below are whole
// blocks further, for W <= 16 a row step stays in the block or moves to the
// next one (halo_row_step).  A step of one column moves 16 bytes within a
// block, or 528 across one (x = 31 | 32 at W = 64); cross bit i: the pixel is
// the last of its block, bit 4 + i: the first.  edge bit i: the pixel is in
// column 0, bit 4 + i: in column W - 1.  A tap that would read column -1 or
// W reads the zero block instead, at the offset it would have had in its own
// block: the half wave's 32 lanes then still hit 32 distinct 16-byte slots
// (one shared zero entry cost a bank conflict on every such read).
template <int W>
struct HaloA {
  int r[4];
  int edge, cross;
};

// halo_addr(p + k W) from a = halo_addr(p) (k = 1, 2), from the bits of a
// that hold p % 32: the step leaves the block when p % 32 + k W >= 32.
template <int W>
__device__ __forceinline__ int halo_row_step(int a, int k) {
  if constexpr (W >= 32) return a + k * (W / 32) * 1024;
  const int d = k * W;                                   // pixels: 8, 16 or 32
  if (d == 32) return a + 1024;
  if (d == 16) return a + 256 + ((a & 256) << 1);        // bit 4 of p: 16 -> next block (+1024 - 256)
  // d == 8: p % 32 >= 24 (bits 3 and 4 of p) -> next block (+1024 - 384)
  return a + 128 + ((a & (a >> 1) & 128) << 2);
}
template <int W, int TN>
__device__ __forceinline__ void halo_abase(int wave, int lane, int RI, HaloA<W>& A) {
  const int h = lane >> 5;
  A.edge = 0;
  A.cross = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = wave * 128 + i * 32 + (lane & 31);
    const int row = m / W, x = m % W;
    const int hp = ((row / RI) * (RI + 2) + row % RI) * W + x;
    A.r[i] = halo_addr(hp, h);
    A.edge |= (x == 0 ? 1 : 0) << i;
    A.edge |= (x == W - 1 ? 1 : 0) << (4 + i);
    A.cross |= ((hp & 31) == 31 ? 1 : 0) << i;
    A.cross |= ((hp & 31) == 0 ? 1 : 0) << (4 + i);
  }
}

// The nine k-steps of the chunk staged at st (B: column j 32 + (lane & 31),
// half h).
template <int W, int TN>
__device__ __forceinline__ void halo_mma(const unsigned char* st, const HaloA<W>& A, int bbase, v16f (&acc)[4][TN]) {
  using G = HaloGeo<W, TN>;
  v8bf fa[2][4], fb[2][TN];
  auto load = [&](int t, int p) {
    const int dy = t / 3, dx = t % 3 - 1;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int off = A.r[i];
      if (W < 32 && dy != 0) {
        // recomputed at each use: kept, the row steps would hold 4-8 more registers
        asm volatile("" : "+v"(off));
        off = halo_row_step<W>(off, dy);
      } else if (dy != 0) {
        off = halo_row_step<W>(off, dy);
      }
      off += dx * 16;
      // a column step crosses a block only inside a 64-pixel row; for
      // W <= 32 the block edges are image edges, which read zeros
      if constexpr (W == 64) {
        if (dx > 0 && ((A.cross >> i) & 1)) off += 512;
        if (dx < 0 && ((A.cross >> (4 + i)) & 1)) off -= 512;
      }
      if (dx != 0 && ((A.edge >> (i + (dx > 0 ? 4 : 0))) & 1)) off = G::HZERO | (off & 1023);
      fa[p][i] = *reinterpret_cast<const v8bf*>(st + off);
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) fb[p][j] = *reinterpret_cast<const v8bf*>(st + bbase + (t * 2 * G::BN + j * 32) * 16);
  };
  load(0, 0);
#pragma unroll
  for (int t = 0; t < 9; ++t) {
    if (t < 8) load(t + 1, (t + 1) & 1);
    __builtin_amdgcn_sched_barrier(0);                 // keep those reads ahead of the MFMAs
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[t & 1][i], fb[t & 1][j], acc[i][j], 0, 0, 0);
  }
}

// Bias, activation and bf16 rounding of a wave's accumulators, packed in
// pairs of rows (e, e + 1).
template <int TN>
__device__ __forceinline__ void halo_round(const ConvArgs& a, const HaloTile& tl, int lane,
                                           const v16f (&acc)[4][TN], uint32_t (&ob)[4][TN][8]) {
  const int ncol = a.cols ? a.ncols : a.Cout;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int nc = tl.n0 + j * 32 + (lane & 31);
    float bv = 0.f;
    if (nc < ncol) {
      if (a.cols) {
        const DeltaCol cd = a.cols[nc];
        bv = a.btab[a.slot0 + cd.slot - a.col_slot0][cd.c];
      } else {
        bv = a.btab[tl.slot][nc];
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 16; e += 2)
        ob[i][j][e >> 1] = f2bf2(act(acc[i][j][e] + bv, a.relu), act(acc[i][j][e + 1] + bv, a.relu));
  }
}

// A wave's 128 rounded pixels into the staging tile Os ([pixel][OLD]) from
// row r0 on.
template <int W, int TN>
__device__ __forceinline__ void halo_stage(bf16_t* Os, int r0, int lane, const uint32_t (&ob)[4][TN][8]) {
  using G = HaloGeo<W, TN>;
  const int h = lane >> 5;
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 16; e += 2) {
        const int r = r0 + i * 32 + (e >> 2) * 8 + h * 4 + (e & 3);
        const uint32_t v = ob[i][j][e >> 1];
        Os[r * G::OLD + j * 32 + (lane & 31)] = (bf16_t)v;
        Os[(r + 1) * G::OLD + j * 32 + (lane & 31)] = (bf16_t)(v >> 16);
      }
}

// band pixel m -> (input xi, image row y, column x); a band's images are RI
// = 2^rsh rows each (RI = H or 512 / W, both powers of two)
template <int W>
__device__ __forceinline__ void halo_pixel(const HaloTile& tl, int rsh, int m, int& xi, int& y, int& x) {
  const int row = m / W;
  x = m % W;
  xi = tl.xi0 + (row >> rsh);
  y = tl.y0 + (row & ((1 << rsh) - 1));
}

template <int W, bool VSKIP>
__device__ __forceinline__ const bf16_t* halo_skip_at(const ConvArgs& a, const HaloTile& tl, int xi, int y, int x,
                                                      int n, int e);

// A fused ADD's shortcut vectors for the output vectors idx = tid + NT k of
// the pixels [m0, m0 + PB) (pixel idx / VPR, channels 8 (idx % VPR)): option
// A, or (IDENT) an identity shortcut read whole.
template <int W, int TN, int PB, bool IDENT>
__device__ __forceinline__ void halo_skip(const ConvArgs& a, const HaloTile& tl, int rsh, int m0, int tid,
                                          v4u (&skipv)[PB * HaloGeo<W, TN>::VPR / HaloGeo<W, TN>::NT]) {
  using G = HaloGeo<W, TN>;
  constexpr int NV = PB * G::VPR / G::NT;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int idx = tid + G::NT * k, m = m0 + idx / G::VPR, n = tl.n0 + (idx % G::VPR) * 8;
    int xi, y, x;
    halo_pixel<W>(tl, rsh, m, xi, y, x);
    skipv[k] = v4u{0u, 0u, 0u, 0u};
    if (n >= a.Cout || xi >= a.nx) continue;
    if constexpr (IDENT) {
      if (a.add_mode == 1) {
        skipv[k] = *reinterpret_cast<const v4u*>(halo_skip_at<W, false>(a, tl, xi, y, x, n, -1));
        continue;
      }
    }
    // option A: the skip subsampled by 2 and zero-padded in channels; with the
    // padding and C_s multiples of 8 a vector is wholly inside or out
    const bf16_t* sp = reinterpret_cast<const bf16_t*>(a.skip.p) +
                       row_at(a.skip.mode, tl.slot, xi, a.nx, a.x0) * a.skip.row_elems;
    const int cs0 = n - (a.Cout - a.Cs) / 2;
    const bf16_t* px = sp + ((int64_t)(2 * y) * a.Ws + 2 * x) * a.Cs;
    if (((a.Cout - a.Cs) / 2) % 8 == 0 && a.Cs % 8 == 0) {
      if (cs0 >= 0 && cs0 < a.Cs) skipv[k] = *reinterpret_cast<const v4u*>(px + cs0);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int cs = cs0 + e;
        if (cs >= 0 && cs < a.Cs) skipv[k][e >> 1] |= (uint32_t)px[cs] << (16 * (e & 1));
      }
    }
  }
}

// Whole output rows of the pixels [m0, m0 + PB) staged in Os (local row
// m - m0), with the ADD's shortcut (add_mode 1 or 2) added in float32 before
// its activation: thread tid stores the vectors idx = tid + NT k.
template <int W, int TN, int PB>
__device__ __forceinline__ void halo_store_rows(const ConvArgs& a, const HaloTile& tl, int rsh, int m0, int tid,
                                                const bf16_t* Os, int add_mode,
                                                const v4u (&skipv)[PB * HaloGeo<W, TN>::VPR / HaloGeo<W, TN>::NT]) {
  using G = HaloGeo<W, TN>;
  constexpr int NV = PB * G::VPR / G::NT;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int idx = tid + G::NT * k, ml = idx / G::VPR, vc = idx % G::VPR;
    const int n = tl.n0 + vc * 8;
    if (n >= a.Cout) continue;
    int xi, y, x;
    halo_pixel<W>(tl, rsh, m0 + ml, xi, y, x);
    if (xi >= a.nx) continue;
    v4u val = *reinterpret_cast<const v4u*>(&Os[ml * G::OLD + vc * 8]);
    if (add_mode) {
      const v4u sv = skipv[k];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float t0 = act(bf2f((bf16_t)val[w]) + bf2f((bf16_t)sv[w]), a.add_relu);
        const float t1 = act(bf2f((bf16_t)(val[w] >> 16)) + bf2f((bf16_t)(sv[w] >> 16)), a.add_relu);
        val[w] = f2bf2(t0, t1);
      }
    }
    const int64_t ro = row_at(a.out_mode, tl.slot, xi, a.nx, a.x0);
    *reinterpret_cast<v4u*>(reinterpret_cast<bf16_t*>(a.out) + ro * a.out_row + ((int64_t)y * W + x) * a.Cout + n) =
        val;
  }
}
// ---- epilogue in two passes for an identity shortcut ----
// Pass P stores the 256 band pixels of M tiles 2P and 2P + 1 of every wave;
// its local pixel ml is band pixel halo_pass_pixel(P, ml).  Pass 0's
// shortcut rows are brought into the stage the last chunk left free by direct
// loads issued with that chunk's MFMAs; pass 1's are loaded into registers
// once pass 0 is staged, under pass 0's stores.
__device__ __forceinline__ int halo_pass_pixel(int P, int ml) { return (ml >> 6) * 128 + P * 64 + (ml & 63); }

// The identity shortcut's channels n .. n + 7 at output pixel (xi, y, x): from
// whole rows, or (VSKIP) read in channel groups, from the shared cache or from
// side plane e of the group (e < 0: unchanged, in the cache).  e is looked up
// once per thread: its channels are the same at every pixel it handles.
template <int W, bool VSKIP>
__device__ __forceinline__ const bf16_t* halo_skip_at(const ConvArgs& a, const HaloTile& tl, int xi, int y, int x,
                                                      int n, int e) {
  if constexpr (VSKIP) {
    const GroupIn& gs = a.gskip;
    const int64_t pix = (int64_t)xi * gs.P + y * W + x;
    return e < 0 ? reinterpret_cast<const bf16_t*>(gs.cache) + pix * gs.C + n
                 : reinterpret_cast<const bf16_t*>(gs.side) + (int64_t)(e - gs.g0) * a.nx * gs.P * 8 + pix * 8;
  }
  return reinterpret_cast<const bf16_t*>(a.skip.p) +
         row_at(a.skip.mode, tl.slot, xi, a.nx, a.x0) * a.skip.row_elems +
         ((int64_t)y * W + x) * a.Cout + n;
}

// Pass 0's shortcut into F as [pixel ml][BN] (16-byte piece p = ml VPR + vc
// at F + 16 p): wave w issues pieces 64 q + lane for q = w, w + 4, ...; a
// lane's vc is lane % VPR, the same as its thread's in the passes.
template <int W, int TN, bool VSKIP>
__device__ __forceinline__ void halo_skip_dma(const ConvArgs& a, const HaloTile& tl, int rsh, int wave, int lane,
                                              unsigned char* F, const bf16_t* zp, int skip_e) {
  using G = HaloGeo<W, TN>;
#pragma unroll
  for (int q = wave; q < 4 * G::VPR; q += 4) {
    const int pc = q * 64 + lane, ml = pc / G::VPR, vc = pc % G::VPR;
    const int n = tl.n0 + vc * 8;
    int xi, y, x;
    halo_pixel<W>(tl, rsh, halo_pass_pixel(0, ml), xi, y, x);
    const bf16_t* src = zp;
    if (n < a.Cout && xi < a.nx) src = halo_skip_at<W, VSKIP>(a, tl, xi, y, x, n, skip_e);
    __builtin_amdgcn_global_load_lds((const void*)src, (lds_void*)(F + q * 1024), 16, 0, 0);
  }
}

// Pass 1's shortcut vectors idx = tid + NT k (pixel ml = idx / VPR) into registers.
template <int W, int TN, bool VSKIP>
__device__ __forceinline__ void halo_skip_pass1(const ConvArgs& a, const HaloTile& tl, int rsh, int tid,
                                                v4u (&sk)[HaloGeo<W, TN>::VPR], int skip_e) {
  using G = HaloGeo<W, TN>;
#pragma unroll
  for (int k = 0; k < G::VPR; ++k) {
    const int idx = tid + G::NT * k, ml = idx / G::VPR, n = tl.n0 + (idx % G::VPR) * 8;
    int xi, y, x;
    halo_pixel<W>(tl, rsh, halo_pass_pixel(1, ml), xi, y, x);
    sk[k] = v4u{0u, 0u, 0u, 0u};
    if (n < a.Cout && xi < a.nx) sk[k] = *reinterpret_cast<const v4u*>(halo_skip_at<W, VSKIP>(a, tl, xi, y, x, n, skip_e));
  }
}

// Bias, activation and bf16 rounding of M tiles 2P and 2P + 1 of a wave's
// accumulators (the other two stay in their registers until their pass), and
// the rounded pixels into Os ([ml][OLD]).
template <int W, int TN>
__device__ __forceinline__ void halo_stage_pass(const ConvArgs& a, const HaloTile& tl, bf16_t* Os, int wave, int P,
                                                int lane, const v16f (&acc)[4][TN]) {
  using G = HaloGeo<W, TN>;
  const int h = lane >> 5;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int nc = tl.n0 + j * 32 + (lane & 31);
    const float bv = nc < a.Cout ? a.btab[tl.slot][nc] : 0.f;
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
#pragma unroll
      for (int e = 0; e < 16; e += 2) {
        const int r = wave * 64 + ii * 32 + (e >> 2) * 8 + h * 4 + (e & 3);
        const v16f& ac = acc[2 * P + ii][j];
        const uint32_t v = f2bf2(act(ac[e] + bv, a.relu), act(ac[e + 1] + bv, a.relu));
        Os[r * G::OLD + j * 32 + (lane & 31)] = (bf16_t)v;
        Os[(r + 1) * G::OLD + j * 32 + (lane & 31)] = (bf16_t)(v >> 16);
      }
  }
}

// Pass P's output rows with the shortcut (from F for pass 0, sk for pass 1)
// added in float32 before its activation.
template <int W, int TN>
__device__ __forceinline__ void halo_store_pass(const ConvArgs& a, const HaloTile& tl, int rsh, int P, int tid,
                                                const bf16_t* Os, const unsigned char* F,
                                                const v4u (&sk)[HaloGeo<W, TN>::VPR]) {
  using G = HaloGeo<W, TN>;
#pragma unroll
  for (int k = 0; k < G::VPR; ++k) {
    const int idx = tid + G::NT * k, ml = idx / G::VPR, vc = idx % G::VPR;
    const int n = tl.n0 + vc * 8;
    if (n >= a.Cout) continue;
    int xi, y, x;
    halo_pixel<W>(tl, rsh, halo_pass_pixel(P, ml), xi, y, x);
    if (xi >= a.nx) continue;
    v4u val = *reinterpret_cast<const v4u*>(&Os[ml * G::OLD + vc * 8]);
    const v4u sv = P == 0 ? *reinterpret_cast<const v4u*>(F + idx * 16) : sk[k];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float t0 = act(bf2f((bf16_t)val[w]) + bf2f((bf16_t)sv[w]), a.add_relu);
      const float t1 = act(bf2f((bf16_t)(val[w] >> 16)) + bf2f((bf16_t)(sv[w] >> 16)), a.add_relu);
      val[w] = f2bf2(t0, t1);
    }
    const int64_t ro = row_at(a.out_mode, tl.slot, xi, a.nx, a.x0);
    *reinterpret_cast<v4u*>(reinterpret_cast<bf16_t*>(a.out) + ro * a.out_row + ((int64_t)y * W + x) * a.Cout + n) =
        val;
  }
}
}  // namespace

// Zero bytes that out-of-image halo pixels and columns past the last read.
static __device__ __attribute__((aligned(16))) v4u g_halo_zero[4] = {};

// Two blocks per CU (at most 80 KB of LDS each).
// V bit 0: the input is read in channel groups (a.gin); bit 1: the identity
// shortcut is (a.gskip).
template <int W, int TN, int V>
__global__ __launch_bounds__(256, 2)
void conv_halo_kernel(ConvArgs a) {
  constexpr bool VIN = (V & 1) != 0, VSKIP = (V & 2) != 0;
  using G = HaloGeo<W, TN>;
  constexpr int BM = G::BM, NT = G::NT, BN = G::BN, OLD = G::OLD, VPR = G::VPR;
  constexpr int NV = BM * VPR / NT;
  constexpr int LDS_B = 2 * G::STAGE > BM * OLD * 2 ? 2 * G::STAGE : BM * OLD * 2;
  __shared__ __attribute__((aligned(16))) unsigned char smem[LDS_B];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  HaloTile tl;
  if (!halo_decode<W, TN>(a, (int)blockIdx.x, tl)) return;   // padding of the order (whole block)
  const int ncol = a.cols ? a.ncols : a.Cout;
  const int RI = a.H < G::TR ? a.H : G::TR;
  const int rsh = 31 - __builtin_clz((unsigned)RI);
  const int npx = (G::TR / RI) * (RI + 2) * W;
  const bf16_t* const zp = reinterpret_cast<const bf16_t*>(g_halo_zero);
  const int nch = a.C / 16;
  // an identity shortcut of the whole tile's rows: the two-pass epilogue
  // (not taken by inputs read in channel groups with a shortcut read whole:
  // slower there, 4.27 against 4.15 ms per width-64 launch on resnet18w)
  const bool split = (!VIN || VSKIP) && !a.cols && !a.pool && a.add_mode == 1;
  static_assert(256 * G::OLD * 2 <= G::STAGE && 256 * G::BN * 2 <= G::STAGE, "a pass fits one stage");
  static_assert(G::STAGE % 1024 == 0 && G::HZERO % 1024 == 0, "stages and zero blocks are 1024-byte aligned");

  HaloSrc<W, TN> hs;
  halo_sources<W, TN, VIN>(a, tl, RI, npx, wave, lane, hs);
  const bf16_t* gb[2] = {nullptr, nullptr};
  int gst[2] = {0, 0};
  int skip_e = -1;
  if constexpr (VSKIP) {
    const int n = tl.n0 + (tid % VPR) * 8;            // the shortcut columns of this thread
    if (n < a.Cout) skip_e = a.gskip.src[tl.slot * (a.gskip.C / 8) + n / 8];
  }
  HaloA<W> A;
  halo_abase<W, TN>(wave, lane, RI, A);
  // the zero blocks of both stages (no load writes them)
  if (tid < 128)
    *reinterpret_cast<v4u*>(smem + (tid >> 6) * G::STAGE + G::HZERO + (tid & 63) * 16) = v4u{0u, 0u, 0u, 0u};
  const int wstep = 9 * a.Cout;                          // chunk-major weight entries per input channel
  const int bbase = G::HALO_B + ((lane >> 5) * BN + (lane & 31)) * 16;
  v16f acc[4][TN];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  if constexpr (VIN) halo_group_bases(a.gin, tl.slot, a.nx, 0, gb, gst);
  halo_fetch<W, TN, VIN>(smem, hs, npx, wave, lane, 0, 0, a.Cout, zp, gb, gst);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  for (int c = 0; c + 1 < nch; ++c) {
    if constexpr (VIN) halo_group_bases(a.gin, tl.slot, a.nx, (c + 1) * 16, gb, gst);
    halo_fetch<W, TN, VIN>(smem + ((c + 1) & 1) * G::STAGE, hs, npx, wave, lane, (c + 1) * 16,
                           (c + 1) * 16 * wstep, a.Cout, zp, gb, gst);
    halo_mma<W, TN>(smem + (c & 1) * G::STAGE, A, bbase, acc);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  }
  // the last chunk, outside the loop: its free stage receives pass 0's shortcut
  if (split) halo_skip_dma<W, TN, VSKIP>(a, tl, rsh, wave, lane, smem + (nch & 1) * G::STAGE, zp, skip_e);
  halo_mma<W, TN>(smem + ((nch - 1) & 1) * G::STAGE, A, bbase, acc);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  // ---- epilogue: bias, activation, bf16 rounding, staged in LDS ----
  if (split) {
    // two passes of 256 pixels through the last chunk's stage
    bf16_t* Os = reinterpret_cast<bf16_t*>(smem + ((nch - 1) & 1) * G::STAGE);
    const unsigned char* F = smem + (nch & 1) * G::STAGE;
    halo_stage_pass<W, TN>(a, tl, Os, wave, 0, lane, acc);
    v4u sk[VPR];                                         // pass 1's shortcut, under pass 0's stores
    halo_skip_pass1<W, TN, VSKIP>(a, tl, rsh, tid, sk, skip_e);
    __syncthreads();
    halo_store_pass<W, TN>(a, tl, rsh, 0, tid, Os, F, sk);
    __syncthreads();
    halo_stage_pass<W, TN>(a, tl, Os, wave, 1, lane, acc);
    __syncthreads();
    halo_store_pass<W, TN>(a, tl, rsh, 1, tid, Os, F, sk);
    return;
  }
  {
    uint32_t ob[4][TN][8];
    halo_round<TN>(a, tl, lane, acc, ob);
    halo_stage<W, TN>(reinterpret_cast<bf16_t*>(smem), wave * 128, lane, ob);
  }
  v4u skipv[NV];
  if (!a.cols && !a.pool && a.add_mode) halo_skip<W, TN, BM, VIN && !VSKIP>(a, tl, rsh, 0, tid, skipv);
  __syncthreads();
  const bf16_t* Os = reinterpret_cast<const bf16_t*>(smem);   // [BM][OLD]
  auto pixel = [&](int m, int& xi, int& y, int& x) { halo_pixel<W>(tl, rsh, m, xi, y, x); };
  if (a.cols) {
    // gathered columns: each column has its own slot and channel
    const int PX = a.pool ? BM / 4 : BM;
    for (int idx = tid; idx < PX * BN; idx += NT) {
      const int nl = idx / PX, q = idx % PX;
      const int nc = tl.n0 + nl;
      if (nc >= ncol) continue;
      int xi, y, x;
      float v;
      if (a.pool) {
        // pooled pixel q: band rows 2 (q / (W/2)) .. +1, columns 2 (q % (W/2)) .. +1
        const int m = 2 * (q / (W / 2)) * W + 2 * (q % (W / 2));
        pixel(m, xi, y, x);
        v = fmaxf(fmaxf(bf2f(Os[m * OLD + nl]), bf2f(Os[(m + 1) * OLD + nl])),
                  fmaxf(bf2f(Os[(m + W) * OLD + nl]), bf2f(Os[(m + W + 1) * OLD + nl])));
        y >>= 1; x >>= 1;
      } else {
        pixel(q, xi, y, x);
        v = bf2f(Os[q * OLD + nl]);
      }
      if (xi >= a.nx) continue;
      const DeltaCol cd = a.cols[nc];
      const int os = a.slot0 + cd.slot - a.col_slot0;
      const int ostride = a.delta_T > 0 ? a.delta_T : a.Cout;
      const int n = a.delta_T > 0 ? cd.t : cd.c;
      const int Wo = a.pool ? W / 2 : W;
      const int64_t ro = row_at(a.out_mode, os, xi, a.nx, a.x0);
      reinterpret_cast<bf16_t*>(a.out)[ro * a.out_row + ((int64_t)y * Wo + x) * ostride + n] = f2bf(v);
    }
    return;
  }
  if (a.pool) {
    for (int idx = tid; idx < (BM / 4) * VPR; idx += NT) {
      const int q = idx / VPR, vc = idx % VPR;
      const int n = tl.n0 + vc * 8;
      if (n >= a.Cout) continue;
      const int m = 2 * (q / (W / 2)) * W + 2 * (q % (W / 2));
      int xi, y, x;
      pixel(m, xi, y, x);
      if (xi >= a.nx) continue;
      // the max of the rounded values is the rounded max (rounding is monotonic)
      const v4u q0 = *reinterpret_cast<const v4u*>(&Os[m * OLD + vc * 8]);
      const v4u q1 = *reinterpret_cast<const v4u*>(&Os[(m + 1) * OLD + vc * 8]);
      const v4u q2 = *reinterpret_cast<const v4u*>(&Os[(m + W) * OLD + vc * 8]);
      const v4u q3 = *reinterpret_cast<const v4u*>(&Os[(m + W + 1) * OLD + vc * 8]);
      v4u o;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        uint32_t r = 0;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int sh = 16 * hh;
          const float f = fmaxf(fmaxf(bf2f((bf16_t)(q0[w] >> sh)), bf2f((bf16_t)(q1[w] >> sh))),
                                fmaxf(bf2f((bf16_t)(q2[w] >> sh)), bf2f((bf16_t)(q3[w] >> sh))));
          r |= (uint32_t)f2bf(f) << sh;
        }
        o[w] = r;
      }
      const int64_t ro = row_at(a.out_mode, tl.slot, xi, a.nx, a.x0);
      *reinterpret_cast<v4u*>(reinterpret_cast<bf16_t*>(a.out) + ro * a.out_row +
                              ((int64_t)(y >> 1) * (W / 2) + (x >> 1)) * a.Cout + n) = o;
    }
    return;
  }
  halo_store_rows<W, TN, BM>(a, tl, rsh, 0, tid, Os, a.add_mode, skipv);
}

int conv_halo_bn(int cout) { return cout <= 32 ? 32 : 64; }

namespace {
template <int W>
hipError_t launch_halo_w(const ConvArgs& a, int bn, int tiles, hipStream_t s) {
  const dim3 grid((unsigned)tiles);
  const int v = (a.gin.cache ? 1 : 0) | (a.gskip.cache ? 2 : 0);
#define MURE_HALO_V(VV)                                                                       \
  if (v == VV) {                                                                             \
    if (bn == 32) hipLaunchKernelGGL((conv_halo_kernel<W, 1, VV>), grid, dim3(256), 0, s, a); \
    else hipLaunchKernelGGL((conv_halo_kernel<W, 2, VV>), grid, dim3(256), 0, s, a);          \
  }
  MURE_HALO_V(0)
  MURE_HALO_V(1)
  MURE_HALO_V(2)
  MURE_HALO_V(3)
#undef MURE_HALO_V
  return hipGetLastError();
}
}  // namespace

hipError_t launch_conv_halo(const ConvArgs& a0, int nslots, hipStream_t s) {
  if (nslots <= 0 || a0.nx <= 0) return hipSuccess;
  if (!conv_halo_fits(a0.H, a0.W, a0.C, a0.kh, a0.kw, a0.stride, a0.pad) || a0.Cout % 8 ||
      a0.out_f32 || a0.add_out_f32 || (a0.pool && a0.add_mode) || a0.vin.chmap)
    return hipErrorInvalidValue;
  if (a0.cols && (a0.in.mode != MODE_CACHE || a0.add_mode || a0.ncols <= 0)) return hipErrorInvalidValue;
  // channel-group reads: pixel indices of the launch's rows stay below 2^31
  if (a0.gin.cache && (a0.cols || !a0.gin.src || a0.gin.C != a0.C || a0.gin.P != a0.H * a0.W ||
                       (int64_t)a0.nx * a0.gin.P >= INT32_MAX))
    return hipErrorInvalidValue;
  if (a0.gskip.cache && (a0.add_mode != 1 || !a0.gskip.src || a0.gskip.C != a0.Cout || a0.gskip.C % 8 ||
                         a0.gskip.P != a0.H * a0.W))
    return hipErrorInvalidValue;
  ConvArgs a = a0;
  if (a.cols) nslots = 1;
  const int TR = 512 / a.W;
  const int ncol = a.cols ? a.ncols : a.Cout;
  const int bn = conv_halo_bn(ncol);
  const int64_t bands = ((int64_t)a.nx * a.H + TR - 1) / TR;
  const int zb = (ncol + bn - 1) / bn;
  const int64_t tiles = (bands + 7) / 8 * 8 * zb * nslots;
  if (tiles >= (1 << 30)) return hipErrorInvalidValue;
  a.bands = (int)bands;
  a.zblocks = zb;
  a.halo_slots = nslots;
  switch (a.W) {
    case 8: return launch_halo_w<8>(a, bn, (int)tiles, s);
    case 16: return launch_halo_w<16>(a, bn, (int)tiles, s);
    case 32: return launch_halo_w<32>(a, bn, (int)tiles, s);
    default: return launch_halo_w<64>(a, bn, (int)tiles, s);
  }
}

}  // namespace mure
