// Kernel argument blocks and host-side launchers of the gfx950 kernels.
//
// Activation tensors are addressed by "row": a row is one (mutant slot,
// input) pair of the current chunk, r = slot * nx + xi with xi in [0, nx).
// A tensor is either a chunk buffer (row r lives at index r) or a prefix-cache
// tensor holding the original model's activation for every input (row r
// reads index x0 + xi, shared by all mutant slots).
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace mure {

enum { MODE_BUF = 0, MODE_CACHE = 1 };

// Unsigned 32-bit division by a divisor fixed at launch, as a multiply-high,
// add and shifts (Granlund and Montgomery, "Division by invariant integers
// using multiplication", PLDI 1994, Figure 4.1): exact for every 32-bit
// dividend.  With l = ceil(log2 d) and mul = floor(2^32 (2^l - d) / d) + 1,
//   t = mulhi(mul, n),  n / d = (t + ((n - t) >> min(l, 1))) >> max(l - 1, 0).
struct DivU32 {
  uint32_t d = 1, mul = 1;
  int sh1 = 0, sh2 = 0;
};

inline DivU32 make_divu32(uint32_t d) {
  DivU32 v;
  if (d == 0) return v;                      // callers never divide by 0; keep d = 1
  int l = 0;
  while (l < 32 && (uint64_t(1) << l) < d) ++l;
  v.d = d;
  v.mul = (uint32_t)(((uint64_t(1) << 32) * ((uint64_t(1) << l) - d)) / d + 1);
  v.sh1 = l < 1 ? l : 1;
  v.sh2 = l > 1 ? l - 1 : 0;
  return v;
}

// Weights of a convolution the halo kernel computes (bf16 3x3, C_in % 16 ==
// 0) are kept chunk-major, [C_in / 16][tap][half][C_out][8], instead of
// [C_out][kh][kw][C_in]: the weight tile of one 16-channel chunk is then 18
// contiguous runs of C_out x 16 bytes.  Index of weight (output channel n,
// tap = ky kw + kx, input channel ci).
__host__ __device__ inline int64_t halo_w_index(int n, int tap, int ci, int Cout) {
  return ((((int64_t)(ci >> 4) * 9 + tap) * 2 + ((ci >> 3) & 1)) * Cout + n) * 8 + (ci & 7);
}

struct TensorArg {
  const void* p = nullptr;
  int mode = MODE_BUF;
  int64_t row_elems = 0;   // elements per row
};

// A consumer's view of the first mutated node's output without materialising
// it per mutant: element (slot, input x, pixel, channel c) is
//   chmap[slot][c] >= 0   the original's channel chmap[slot][c] (prefix cache),
//   chmap[slot][c] == -1  zero (effect block),
//   chmap[slot][c] <= -2  recomputed channel t = -2 - chmap[slot][c], read from
//                         the compact delta rows delta[r][pixel][t] (r = chunk row).
struct VirtualIn {
  const void* cache = nullptr;           // [N][H][W][C]
  const int32_t* chmap = nullptr;        // [chunk slots][C]; nullptr: not virtual
  const void* delta = nullptr;           // [chunk rows][H*W][T]
  int C = 0, HW = 0, T = 0;
};

// A bf16 tensor read in 8-channel groups: the first mutated node's output as
// the halo kernel's input or fused shortcut, with only each slot's changed
// groups materialised.  Group g of launch slot s at input row xi (relative to
// the launch's first input), pixel p: when src[s * C / 8 + g] = e >= 0, side
// plane e - g0 at element (xi * P + p) * 8; otherwise cache element
// (xi * P + p) * C + 8 g (cache points at the launch's first input).
struct GroupIn {
  const void* cache = nullptr;           // nullptr: not in use
  const int32_t* src = nullptr;          // [slots][C / 8]
  const void* side = nullptr;            // [planes][nx][P][8]
  int g0 = 0, C = 0, P = 0;
};

// Build the side planes of a GroupIn: plane e holds group ent[2e+1] of slot
// ent[2e] through that slot's channel map (>= 0: cached channel, -1: zero,
// <= -2: compact delta channel -2 - map, in delta row (slot - slot0) nx + xi).
struct GroupPatchArgs {
  const void* cache = nullptr;           // the launch's first input: [nx][P][C]
  const int32_t* chmap = nullptr;        // [slots][C], indexed by ent's slot
  const void* delta = nullptr;           // [(slots - slot0) * nx][P][T]
  const int32_t* ent = nullptr;          // [n_ent][2]: (slot, group)
  void* side = nullptr;                  // [n_ent][nx][P][8]
  int n_ent = 0, nx = 0, P = 0, C = 0, T = 0, slot0 = 0;
};

// One gathered output column of the delta at the first mutated node: output
// channel `c` of mutant slot `slot - col_slot0` (relative to the launch's
// slot0).  A delta launch shares the cached input among all its columns and
// computes only the channels the mutants' records changed; column results are
// stored as compact delta channel `t` (delta_T > 0) or as channel c of the
// slot's full row.
struct DeltaCol {
  int slot, c, t, pad;
};

// CONV2D / DENSE (a DENSE layer is a 1x1 convolution over a 1x1xC_in input).
struct ConvArgs {
  TensorArg in;
  VirtualIn vin;                         // used instead of `in` when vin.chmap != nullptr
  void* out = nullptr;
  int out_mode = MODE_BUF;
  int64_t out_row = 0;
  int out_f32 = 0;                       // 1: store float32 (network output)
  const void* const* wtab = nullptr;     // [slots] weights [C_out][kh][kw][C_in]
  const float* const* btab = nullptr;    // [slots] bias [C_out]
  int slot0 = 0;                         // first slot of this launch (rows start at slot0*nx)
  int nx = 0, x0 = 0;
  int H = 0, W = 0, C = 0;               // input geometry
  int Hc = 0, Wc = 0;                    // convolution output before pooling
  int Hp = 0, Wp = 0;                    // stored output
  int Cout = 0, kh = 1, kw = 1, stride = 1, pad = 0, relu = 0, pool = 0;
  int K = 0;                             // kh*kw*C
  int P = 0;                             // GEMM rows per input
  // fused ADD node after this convolution (conv_b of a residual block; its
  // own output is rounded first, then out = ReLU?(conv + s(skip)) is stored
  // as the ADD node's output): 0 none, 1 identity shortcut, 2 option A
  int add_mode = 0, add_relu = 0, add_out_f32 = 0;
  TensorArg skip;
  int Hs = 0, Ws = 0, Cs = 0;            // skip geometry
  int tile = 0;                          // tiled kernel's block shape (0 automatic)
  // halo kernel only: input / identity shortcut read in 8-channel groups
  GroupIn gin, gskip;
  // gathered-column delta (cols != nullptr): ncols columns instead of C_out
  // channels per slot; the input must be slot independent (prefix cache)
  const DeltaCol* cols = nullptr;
  int ncols = 0, delta_T = 0, col_slot0 = 0;
  // filled by the launchers: dividers by P, P/4, Wp, Wc, H*W, C, kw and the
  // padded image size; the halo kernel's band count and column blocks per
  // band (XCD-aware order)
  DivU32 dP, dPq, dWp, dWc, dHW, dC, dKW, dImg;
  int bands = 0, zblocks = 1, halo_slots = 1;
  int big_gx = 1, big_gz = 1, big_tiles = 0;            // conv_big: row tiles, column blocks, all tiles
};

// DENSE on MFMA: out[r][n] = sum_k in[r][k] * W[n][k] + b[n] (k in increasing
// steps), optional ReLU; optionally fused with the kill reduction when one
// block column covers every class.
struct DenseArgs {
  TensorArg in;                          // row_elems = K
  VirtualIn vin;                         // used instead of `in` when vin.chmap != nullptr
  void* out = nullptr;
  int out_mode = MODE_BUF, out_f32 = 0, write_out = 1;
  const void* const* wtab = nullptr;
  const float* const* btab = nullptr;
  int slot0 = 0, nx = 0, x0 = 0, K = 0, Cout = 0, relu = 0;
  // fused kill
  int do_kill = 0;
  const int32_t* slot_mutant = nullptr;
  const int32_t* label = nullptr;
  const uint8_t* orig_ok = nullptr;
  uint64_t* kill_words = nullptr;
  int64_t nwords = 0;
  unsigned long long* nonfinite = nullptr;
  float* logits_out = nullptr;
  // gathered-column delta, as in ConvArgs (no kill, no virtual input)
  const DeltaCol* cols = nullptr;
  int ncols = 0, delta_T = 0, col_slot0 = 0;
};

// CONV2D with tiny C_out on the vector ALU, one output position per thread.
// ch_off/ch_list (optional) restrict each slot to a list of output channels:
// slot sl computes channels ch_list[ch_off[sl] .. ch_off[sl+1]).
struct ValuArgs {
  TensorArg in;
  void* out = nullptr;
  int out_mode = MODE_BUF, out_f32 = 0;
  int64_t out_row = 0;
  const void* const* wtab = nullptr;
  const float* const* btab = nullptr;
  int slot0 = 0, nslots = 0, nx = 0, x0 = 0;
  int H = 0, W = 0, C = 0, Hp = 0, Wp = 0;
  int Cout = 0, kh = 1, kw = 1, stride = 1, pad = 0, relu = 0, pool = 0, K = 0;
  const int32_t* ch_off = nullptr;
  const int32_t* ch_list = nullptr;
  int delta_T = 0;                       // > 0: write channel t of the list to the compact
                                         // delta row out[r][q][t] (out_row = Hp*Wp*delta_T)
};

// Depthwise CONV2D: output channel c filters input channel c with its own
// kh x kw taps.  ch_off/ch_list (optional) restrict slot sl to the channels
// ch_list[ch_off[sl] .. ch_off[sl+1]) (the delta at the first mutated layer),
// written as compact delta entries (delta_T > 0) or into full rows.
struct DwArgs {
  TensorArg in;
  void* out = nullptr;
  int out_mode = MODE_BUF, out_f32 = 0;
  int64_t out_row = 0;
  const void* const* wtab = nullptr;     // [slots] weights [C][kh][kw]
  const float* const* btab = nullptr;
  int slot0 = 0, nslots = 0, nx = 0, x0 = 0;
  int H = 0, W = 0, C = 0, Ho = 0, Wo = 0;
  int kh = 3, kw = 3, stride = 1, pad = 0, relu = 0;
  const int32_t* ch_off = nullptr;
  const int32_t* ch_list = nullptr;
  int delta_T = 0;
};

// Sequence layers (float32): EMBED out[row][t][d] = W[d][token] for T tokens
// of a row (V = vocabulary, D = width); LSTM over T steps of [row][T][D] with
// H units, weights [H][4][D + H + 1] per slot, output every step (seq) or the
// last one.
struct SeqArgs {
  TensorArg in;
  void* out = nullptr;
  int out_mode = MODE_BUF, out_f32 = 0;
  int64_t out_row = 0;
  const void* const* wtab = nullptr;
  int slot0 = 0, nslots = 0, nx = 0, x0 = 0;
  int T = 0, D = 0, H = 0, V = 0, seq = 0;
};

struct AddArgs {
  TensorArg a, s;
  void* out = nullptr;
  int out_mode = MODE_BUF, out_f32 = 0;
  int nx = 0, x0 = 0;
  int64_t rows = 0;
  int H = 0, W = 0, C = 0;               // output (= in[0]) geometry
  int Hs = 0, Ws = 0, Cs = 0;            // in[1] geometry
  int shortcut = 0, relu = 0;
};

struct GapArgs {
  TensorArg in;
  void* out = nullptr;
  int out_mode = MODE_BUF, out_f32 = 0;
  int nx = 0, x0 = 0;
  int64_t rows = 0;
  int P = 0, C = 0;
};

struct PatchArgs {                       // channel patch of node mmi for NEB/NS mutants
  const void* cache = nullptr;           // original output of mmi, all inputs
  void* out = nullptr;                   // chunk buffer
  const int32_t* chmap = nullptr;        // [patch slots][C]: source channel or -1
  int slot0 = 0;                         // first slot of this launch
  int chmap_slot0 = 0;                   // chmap row of slot0
  int nx = 0, x0 = 0, nslots = 0;
  int P = 0, C = 0, esize = 2;
};

struct KillArgs {
  const float* logits = nullptr;         // chunk buffer [rows][C]
  int C = 0, nx = 0, x0 = 0, nslots = 0, slot0 = 0;
  const int32_t* slot_mutant = nullptr;  // global mutant id of each slot of the group
  const int32_t* label = nullptr;        // [N]
  const uint8_t* orig_ok = nullptr;      // [N] argmax original == label
  uint64_t* kill_words = nullptr;        // [M][nwords]
  int64_t nwords = 0;
  unsigned long long* nonfinite = nullptr;
  float* logits_out = nullptr;           // optional [N][C] copy (single-slot runs)
};

struct LabelArgs {
  const float* logits = nullptr;         // [N][C]
  int64_t N = 0;
  int C = 0;
  const int32_t* given = nullptr;        // optional [N]
  int32_t* label = nullptr;
  uint8_t* ok = nullptr;
  unsigned long long* class_mask = nullptr;   // [ceil(C/64)]
  unsigned long long* nonfinite = nullptr;
};

struct ScoreArgs {
  const uint64_t* kill_words = nullptr;
  int64_t nwords = 0;
  int64_t N = 0;
  const int32_t* label = nullptr;
  int mask_words = 0;
  int64_t* kills = nullptr;                   // [M]
  unsigned long long* masks = nullptr;        // [M][mask_words]
};

struct CowArgs {                           // one copy-on-write parameter copy
  const void* w_src; void* w_dst;
  const float* b_src; float* b_dst;
  int c_out; int64_t fan_in;
  int64_t rs, ks;                          // element strides of a neuron's row and of k (EMBED: 1, c_out)
  int halo_c;                              // > 0: chunk-major halo weights with this C_in (rs, ks unused)
  int rec0, rec1;                          // records [rec0, rec1) in the device record table
};

struct DevRecord { int op, neuron, partner, pad; int64_t noise_off, scratch_off; };

// launchers (return the launch status)
hipError_t launch_conv(const ConvArgs& a, int nslots, int dtype, hipStream_t s);
hipError_t launch_conv_lds(const ConvArgs& a, int nslots, hipStream_t s);
hipError_t launch_conv_big(const ConvArgs& a, int nslots, hipStream_t s);
hipError_t launch_conv_halo(const ConvArgs& a, int nslots, hipStream_t s);
hipError_t launch_dense(const DenseArgs& a, int nslots, int dtype, hipStream_t s);
hipError_t launch_valu(const ValuArgs& a, int dtype, hipStream_t s);
hipError_t launch_dw(const DwArgs& a, int dtype, hipStream_t s);
hipError_t launch_embed(const SeqArgs& a, hipStream_t s);
hipError_t launch_lstm(const SeqArgs& a, hipStream_t s);
hipError_t launch_add(const AddArgs& a, int dtype, hipStream_t s);
hipError_t launch_gap(const GapArgs& a, int dtype, hipStream_t s);
hipError_t launch_patch(const PatchArgs& a, hipStream_t s);
hipError_t launch_kill(const KillArgs& a, hipStream_t s);
hipError_t launch_labels(const LabelArgs& a, hipStream_t s);
hipError_t launch_score(const ScoreArgs& a, int n_mutants, hipStream_t s);
hipError_t launch_group_patch(const GroupPatchArgs& a, hipStream_t s);
hipError_t launch_cow(const CowArgs* d_args, int n_copies, const DevRecord* d_recs,
                      const float* d_noise, int dtype, hipStream_t s);
hipError_t launch_copy_rows(const TensorArg& src, void* dst, int64_t rows, int nx, int x0,
                            int esize, hipStream_t s);
hipError_t launch_zero_u64(uint64_t* p, int64_t n, hipStream_t s);   // p[0 .. n) = 0

// Device address of this GPU's scratch array of MURE_NOALLOC_SCRATCH_BYTES
// (the allocation-free run_mutants); looked up once per device, which must be
// current.
hipError_t noalloc_scratch(int device, void** out);

}  // namespace mure
