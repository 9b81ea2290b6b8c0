// Host planner for memoized mutation testing (no HIP dependency).
//
// Graph validation and shape inference, the dependence graph (Algorithm 2,
// given explicitly by the node descriptors), each mutant's mutated layers,
// earliest mutated layer mmi and memoization boundary K (Algorithm 1;
// Section 4), the clustering of mutants (grouped by mmi, which determines K),
// the prefix-cache set, the per-mutant channel patches at mmi, and the MAC
// ledger of Section 4.2 (Lemma 4).
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace mure {

enum Kind {
  K_INPUT = 0, K_DENSE = 1, K_CONV = 2, K_ADD = 3, K_GAP = 4, K_FLATTEN = 5, K_DWCONV = 6,
  K_EMBED = 7, K_LSTM = 8
};
enum Op { OP_GF = 0, OP_NEB = 1, OP_NAI = 2, OP_NS = 3, OP_WS = 4 };
enum DType { DT_F32 = 0, DT_BF16 = 1 };

struct Node {
  int kind = 0, n_in = 0, in[2] = {-1, -1};
  int c_in = 0, c_out = 0, kh = 1, kw = 1, stride = 1, pad = 0;
  int relu = 0, maxpool = 0, shortcut = 0, seq = 0;
  // derived
  int H = 0, W = 0, C = 0;        // output shape (after pool)
  int Hc = 0, Wc = 0;             // convolution output before pooling
  int inH = 0, inW = 0, inC = 0;  // shape of in[0]
  int64_t fan_in = 0;             // weights per neuron
  int64_t macs = 0;               // multiply-accumulates per input
  bool weighted() const {
    return kind == K_DENSE || kind == K_CONV || kind == K_DWCONV || kind == K_EMBED || kind == K_LSTM;
  }
  int64_t out_elems() const { return (int64_t)H * W * C; }
  int64_t n_weights() const { return weighted() ? (int64_t)c_out * fan_in : 0; }
};

struct Graph {
  int dtype = DT_F32;
  std::vector<Node> nodes;
  int out() const { return (int)nodes.size() - 1; }
  int classes() const { return nodes.back().C; }
  int64_t full_macs() const;
  // bytes per input of node v's activation as stored (the output node is float32)
  int64_t act_bytes(int v) const;
};

// Validates `nodes` (topological order, shapes, kind-specific fields) and
// fills the derived fields.  Returns "" on success, else a message.
std::string build_graph(Graph& g, int in_h, int in_w, int in_c, int dtype);

struct Record {
  int mutant, op, layer, neuron, partner;
  int64_t noise_off, noise_len;   // into the concatenated parameter array (noise or
                                  // permutation, 4 bytes per entry)
  int64_t scratch_off = 0;        // weight shuffle: row scratch in the same array
};

// Kernel family of a CONV2D/DENSE node -- a pure function of its shape, so
// every launch that computes a node (original forward, recompute at mmi,
// suffix) uses the same accumulation order.
enum Family {
  FAM_DENSE = 0,   // dense GEMM on MFMA
  FAM_VALU = 1,    // tiny C_out: per-output fused multiply-add chains (vector ALU)
  FAM_LDS = 2,     // fp32 conv whose padded input image and weights fit in LDS
  FAM_GEMM = 3,    // implicit GEMM with a scalar im2col gather (any shape)
  FAM_BIG = 4,     // bf16 tiled implicit GEMM with 16-byte gathers (C_in % 8 == 0)
  FAM_DW = 5,      // depthwise convolution (per-channel taps on the vector ALU)
  FAM_EMBED = 6,   // embedding lookup (a gather)
  FAM_LSTM = 7,    // LSTM recursion: per step one MFMA GEMM over [x_t, h, 1], gates on the VALU
  FAM_HALO = 8     // bf16 3x3 stride-1 conv, operands from LDS halo and weight tiles per 16-channel chunk
};
constexpr int N_FAMILIES = 9;
// Halo convolution: 512-pixel bands of TR = 512 / W image rows (the bands
// never straddle two images); a band's halo -- its rows plus the row above
// and below, per packed image -- holds at most conv_halo_cap(W) pixels, the
// halo of square images of that width.
constexpr int conv_halo_cap(int W) { return W == 64 ? 640 : W == 32 ? 576 : W == 16 ? 576 : 640; }
inline bool conv_halo_fits(int H, int W, int C, int kh, int kw, int stride, int pad) {
  if (kh != 3 || kw != 3 || stride != 1 || pad != 1 || C % 16 || C <= 0 || H % 2) return false;
  if (W != 8 && W != 16 && W != 32 && W != 64) return false;
  const int TR = 512 / W;
  if (H % TR && TR % H) return false;
  const int RI = H < TR ? H : TR, IMGS = TR / RI;
  return IMGS * (RI + 2) * W <= conv_halo_cap(W) && (int64_t)9 * C <= (1 << 20);
}
// LSTM kernel: units a multiple of 16, at most 64; LDS for the weights
// (k-major, row stride 4H + 16) and a 64-row step tile
constexpr int lstm_kpad(int d, int h) { return (d + h + 1 + 3) / 4 * 4; }
constexpr int lstm_ka(int d, int h) { const int k = lstm_kpad(d, h); return (k / 4) % 2 ? k : k + 4; }
constexpr int64_t lstm_lds_bytes(int d, int h) {
  return ((int64_t)lstm_kpad(d, h) * (4 * h + 16) + 64LL * lstm_ka(d, h)) * 4;
}
// Wide LSTM kernel (layers whose weights do not fit in LDS): per lane the
// weights of KS k-steps of 4 in registers, KS = ceil((D + H + 1) / 4) rounded
// up to a multiple of 4 (8 .. 52); LDS for two step tiles [KS][64][4].
constexpr int LSTM_WIDE_KS = 52;
constexpr int lstm_wide_ks(int d, int h) { return ((d + h + 1 + 3) / 4 + 3) / 4 * 4 < 8 ? 8 : ((d + h + 1 + 3) / 4 + 3) / 4 * 4; }
constexpr int64_t lstm_wide_lds_bytes(int d, int h) { return 2LL * lstm_wide_ks(d, h) * 256 * 4; }
inline bool lstm_uses_wide(int d, int h) { return lstm_lds_bytes(d, h) > 64 * 1024; }
inline bool lstm_wide_fits(int d, int h) {
  return d % 4 == 0 && lstm_wide_ks(d, h) <= LSTM_WIDE_KS && lstm_wide_lds_bytes(d, h) <= 160 * 1024;
}
int node_family(const Graph& g, int v);

// Launch geometry shared by the planner (family choice) and the kernels.
// VALU convolution: rows per block and LDS bytes (zero-padded fp32 images of
// those rows + the fp32 weights of every output channel).
inline int valu_rows(int Q) { int r = (1024 + Q - 1) / Q; return r < 1 ? 1 : (r > 8 ? 8 : r); }
inline int64_t valu_lds_bytes(int inH, int inW, int inC, int pad, int Q, int c_out, int64_t K) {
  return (int64_t)valu_rows(Q) * (inH + 2 * pad) * (inW + 2 * pad) * inC * 4 + (int64_t)c_out * K * 4;
}
// LDS convolution: images a block may touch for 256 GEMM rows of P per input.
// images a 256-row piece spans: exactly 256 / P when P divides 256 (pieces
// then start at image boundaries), else at most ceil(256 / P) + 1
inline int conv_lds_nimg_cap(int P) {
  return P >= 256 ? 2 : 256 % P == 0 ? 256 / P : (256 + P - 1) / P + 1;
}
inline int conv_lds_bn(int c_out) { return c_out <= 16 ? 16 : c_out <= 32 ? 32 : 64; }
// floats per k row of the LDS weight tile [kpad][kst]: the 4 k rows one MFMA
// reads land in distinct bank quarters
inline int conv_lds_kst(int bn) { return bn == 16 ? 16 : bn + 16; }
inline int64_t conv_lds_bytes(int inH, int inW, int inC, int pad, int P, int c_out, int64_t K) {
  // weights and offsets carry 8 and 16 rows of zero padding past kpad: the
  // software-pipelined k loop reads up to weight row kpad + 7 and offset
  // kpad + 15
  const int64_t kpad = (K + 7) / 8 * 8;
  return ((int64_t)conv_lds_nimg_cap(P) * (inH + 2 * pad) * (inW + 2 * pad) * inC +
          (int64_t)conv_lds_kst(conv_lds_bn(c_out)) * (kpad + 8)) * 4 + (kpad + 16) * 4 +
         (int64_t)inC * 4;
}

struct MutantPlan {
  int mmi = -1;                 // -1: identity mutant (no records)
  int group = -1;
  int slot = -1;                // position inside its group
  std::vector<int> layers;      // mu(M'), ascending
  std::vector<int> K;           // memoization boundary, ascending
  bool recompute = false;       // a fuzz/inverse record at mmi: recompute node mmi
  std::vector<int> chmap;       // output channel c of mmi <- original channel chmap[c]
                                // (-1 = zero); identity for recompute mutants; size c_out(mmi)
  int64_t touched = 0;          // channels of mmi changed by fuzz/inverse records
  std::vector<int> touched_list;  // recompute mutants: every channel of mmi any record
                                  // changes (fuzz/inverse neurons, blocked, switched), ascending
};

// Copy-on-write parameter copy of one (mutant, layer).
struct CowCopy {
  int mutant, layer;
  std::vector<int> records;     // indices into the record array, in order
};

struct Group {
  int mmi = -1;
  std::vector<int> K;
  std::vector<int> mutants;     // global ids; recompute mutants first
  int n_recompute = 0;
  bool delta = false;           // recompute only the touched channels of mmi (VALU family)
  bool virt = false;            // consumers read mmi's output through per-slot channel maps
                                // (cache + compact delta rows); mmi is never materialised
  int T = 0;                    // channels per delta row (virt): max touched list (delta)
                                // or C_out (whole-node recompute)
  std::vector<int> vchmap;      // virt, vhalo: [slot][C_out] channel map (-2-t = delta channel t)
  bool vhalo = false;           // the halo kernel reads mmi's output in 8-channel groups:
                                // each slot's changed groups materialised, the others
                                // from the cache (needs the ADD fused, see fused_add_of)
};

struct Plan {
  int n_mutants = 0;
  std::vector<MutantPlan> mutants;
  std::vector<Group> groups;
  std::vector<CowCopy> cows;
  std::vector<int> cache_nodes;  // nodes whose original activations are cached
  int64_t n_identity = 0;
  // ledger, per input
  int64_t macs_vanilla = 0, macs_memoized = 0, macs_algorithmic = 0, macs_executed = 0;
};

// The ADD node fused into convolution v's epilogue (v's only reader, reading
// it as in[0]), or -1.
int fused_add_of(const Graph& g, int v);

// Memoization boundary K of a first mutated layer (Algorithm 1 / Section 4).
std::vector<int> boundary(const Graph& g, int mmi);

// Validates records and builds the plan.  Returns "" or a message.
// vanilla: no memoization -- every mutant runs from the first layer after
// the input (exhaustive mutation testing, the paper's baseline).
std::string build_plan(const Graph& g, int n_mutants, const std::vector<Record>& recs,
                       Plan& plan, bool vanilla = false);

}  // namespace mure
