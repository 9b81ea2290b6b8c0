// C ABI of the library: context, state machine, device memory, and the
// executor that runs the original model (filling the prefix cache) and every
// mutant's suffix over chunks of (mutant slots x inputs).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <map>
#include <memory>
#include <new>
#include <set>
#include <stdexcept>
#include <string>
#include <thread>
#include <vector>

#include "../../include/mure.h"
#include "kernels.hpp"
#include "plan.hpp"

using namespace mure;

namespace {

thread_local std::string g_create_error;

struct DevBuf {
  void* p = nullptr;
  size_t bytes = 0;
  DevBuf() = default;
  DevBuf(const DevBuf&) = delete;
  DevBuf& operator=(const DevBuf&) = delete;
  ~DevBuf() { release(); }
  void release() {
    if (p) (void)hipFree(p);
    p = nullptr;
    bytes = 0;
  }
  hipError_t alloc(size_t n) {
    release();
    if (n == 0) return hipSuccess;
    hipError_t e = hipMalloc(&p, n);
    if (e == hipSuccess) bytes = n;
    else p = nullptr;
    return e;
  }
  // grow-only: keep the allocation when it is large enough (no free/malloc
  // churn between calls)
  hipError_t ensure(size_t n) {
    if (n <= bytes && p) return hipSuccess;
    return alloc(n < 256 ? 256 : n);
  }
  template <typename T> T* as() const { return reinterpret_cast<T*>(p); }
};

// Page-locked host staging (hipHostMalloc), grow-only: uploads from it are
// plain DMA transfers instead of the runtime's pageable-copy path.
struct PinnedBuf {
  void* p = nullptr;
  size_t bytes = 0;
  PinnedBuf() = default;
  PinnedBuf(const PinnedBuf&) = delete;
  PinnedBuf& operator=(const PinnedBuf&) = delete;
  ~PinnedBuf() {
    if (p) (void)hipHostFree(p);
  }
  hipError_t ensure(size_t n) {
    if (n <= bytes && p) return hipSuccess;
    if (p) (void)hipHostFree(p);
    p = nullptr;
    bytes = 0;
    hipError_t e = hipHostMalloc(&p, n < 4096 ? 4096 : n, hipHostMallocDefault);
    if (e == hipSuccess) bytes = n < 4096 ? 4096 : n;
    else p = nullptr;
    return e;
  }
};

// Liveness-based placement of per-row activation buffers: offsets in bytes
// per row; a buffer is reused once every reader of its previous owner ran.
struct Placement {
  std::map<int, int64_t> offset;   // node -> byte offset per row
  int64_t peak = 0;                // bytes per row
};

Placement place_buffers(const Graph& g, const std::vector<int>& nodes, const std::set<int>& external,
                        const std::map<int, int>& fused = {}) {
  // nodes: executed in this order; external: nodes whose output lives
  // elsewhere; fused: conv_b -> ADD pairs run as one launch at conv_b's step,
  // so the ADD's buffer is placed at that step (conv_b itself has none)
  std::map<int, int> last_use;
  for (int v : nodes) {
    for (int k = 0; k < g.nodes[v].n_in; ++k) last_use[g.nodes[v].in[k]] = v;
  }
  struct Blk { int64_t off, size; int owner; };
  std::vector<Blk> blocks;
  Placement pl;
  const int out = g.out();
  std::set<int> placed;
  auto place = [&](int v) {
    const int64_t need = (g.act_bytes(v) + 255) / 256 * 256;
    int best = -1;
    for (size_t i = 0; i < blocks.size(); ++i)
      if (blocks[i].owner < 0 && blocks[i].size >= need && (best < 0 || blocks[i].size < blocks[best].size))
        best = (int)i;
    if (best < 0) {
      blocks.push_back({pl.peak, need, v});
      pl.peak += need;
      best = (int)blocks.size() - 1;
    } else {
      blocks[best].owner = v;
    }
    pl.offset[v] = blocks[best].off;
    placed.insert(v);
  };
  for (int v : nodes) {
    // free blocks whose owner is no longer needed by v or later nodes
    for (Blk& b : blocks) {
      if (b.owner < 0) continue;
      auto it = last_use.find(b.owner);
      const int lu = (b.owner == out) ? 1 << 30 : (it == last_use.end() ? -1 : it->second);
      if (lu < v) b.owner = -1;
    }
    auto f = fused.find(v);
    if (f != fused.end()) {
      if (!external.count(f->second)) place(f->second);
      continue;
    }
    if (external.count(v) || placed.count(v)) continue;
    place(v);
  }
  return pl;
}

}  // namespace

struct mure_ctx {
  int device = -1;
  bool plan_only = false;
  hipStream_t stream = nullptr;
  hipEvent_t ev0 = nullptr, ev1 = nullptr;
  std::string err;
  int state = 0;   // 0 created, 1 model loaded, 2 mutants applied, 3 original run
  Graph g;
  bool have_graph = false;
  std::vector<std::unique_ptr<DevBuf>> d_w, d_b;     // original parameters per node
  // mutants
  Plan plan;
  std::vector<Record> recs;
  DevBuf d_cow;                                       // copy-on-write parameters
  // the applied mutants' device tables, uploaded as one block: pointer
  // tables, slot/touched-list ints, channel maps, delta columns, copy-on-write
  // arguments, device records and noise
  DevBuf d_apply;
  PinnedBuf h_apply;
  const void** tables = nullptr;
  int32_t* slotv = nullptr;
  int32_t* chmapv = nullptr;
  DeltaCol* colv = nullptr;
  struct GroupTabs {
    std::map<int, int64_t> w, b;                      // node -> offset (in pointers) into tables
    int64_t slot_mutant = 0;                          // offset (int32) into slotv
    int64_t chmap = 0;                                // offset (int32) into chmapv: [slots][C]
    int64_t choff = 0;                                // offset (int32) into slotv: touched-list
                                                      // offsets of the recompute slots (+1)
    int64_t vchmap = 0;                               // offset (int32) into chmapv: virtual maps
    int64_t cols = 0;                                 // offset (DeltaCol) into colv
    std::vector<int64_t> colbeg;                      // first column of each recompute slot (+1)
    int64_t vgsrc = 0;                                // vhalo: offset (int32) into chmapv of the
                                                      // [slots][C/8] side-plane table (-1: cache)
    int64_t vgent = 0;                                // vhalo: offset (int32) into chmapv of the
                                                      // (slot, group) entries, one per side plane
    std::vector<int64_t> vgbeg;                       // vhalo: first entry of each slot (+1)
  };
  std::vector<GroupTabs> gtabs;
  std::map<int, int64_t> orig_w, orig_b;              // node -> offset of 1-entry original tables
  DevBuf d_given;                                     // ground-truth labels
  // prefix cache and original results
  int64_t N = 0;
  std::map<int, std::unique_ptr<DevBuf>> cache;
  DevBuf d_logits, d_label, d_ok, d_classmask, d_nonfinite;
  int64_t n_labels = 0;
  // run_mutants scratch
  DevBuf d_ws, d_kill, d_kills, d_masks;
  DevBuf d_side;                                      // changed channel groups (vhalo clusters)
  int64_t group_reads = 1;                            // option "group_reads"
  void* scratch = nullptr;                            // this GPU's scratch array (noalloc entry)
  // options
  int64_t max_ws_mb = 65536;
  int64_t max_device_mb = 0;                          // 0: no cap on model + copies + prefix cache
  int64_t cow_bytes = 0;                              // copy-on-write pool of the applied mutants
  int64_t chunk_inputs = 0;
  int64_t fused = 1;
  int64_t kernel_timing = 0;
  int64_t conv_tile = 0;
  int64_t vanilla = 0;
  std::vector<hipEvent_t> tevents;                    // pairs around timed launches
  std::vector<int> tevent_family;                     // kernel family of each timed pair
  std::vector<char> tevent_mmi;                       // ... and whether it computed a first mutated node
  size_t tevents_used = 0;
  mure_stats stats{};

  mure_status fail(mure_status s, const std::string& m) {
    err = m;
    return s;
  }
  mure_status dev_fail(hipError_t e, const char* what) {
    err = std::string(what) + ": " + hipGetErrorString(e);
    return e == hipErrorOutOfMemory ? MURE_E_NOMEM : MURE_E_DEVICE;
  }
};

#define HIPTRY(expr)                                  \
  do {                                                \
    hipError_t e_ = (expr);                           \
    if (e_ != hipSuccess) return ctx->dev_fail(e_, #expr); \
  } while (0)

namespace {

int64_t esize_of(const Graph& g, int v) { return (v == g.out() || g.dtype == DT_F32) ? 4 : 2; }

// device bytes of the original parameters
int64_t model_bytes(const Graph& g) {
  const int64_t es = g.dtype == DT_F32 ? 4 : 2;
  int64_t b = 0;
  for (const Node& n : g.nodes)
    if (n.weighted()) b += n.n_weights() * es + (int64_t)n.c_out * 4;
  return b;
}


// Tensor reference of node p for the executor.
struct Where {
  const void* p;
  int mode;
};

// Extra arguments of a weighted-node launch.
struct Extra {
  const int32_t* ch_off = nullptr;    // per-slot channel lists (VALU delta at mmi)
  const int32_t* ch_list = nullptr;
  int delta_T = 0;                    // write compact delta rows of delta_T channels
  const DeltaCol* cols = nullptr;     // gathered-column delta at mmi (MFMA families)
  int ncols = 0, col_slot0 = 0;
  int64_t exec_macs = -1;             // MACs the launch executes, when not slots * rows * node
  int64_t delta_channels = -1;        // channels a per-slot channel-list delta computes
  const VirtualIn* vin = nullptr;     // read the first mutated node's output virtually
  const GroupIn* gin = nullptr;       // ... in 8-channel groups (halo kernel)
  const GroupIn* gskip = nullptr;     // the fused ADD's shortcut, in 8-channel groups
  int fuse_add = -1;                  // ADD node fused into this convolution's epilogue
  Where skip{nullptr, MODE_BUF};      // that ADD's shortcut input
  const KillArgs* kill = nullptr;     // fuse the kill reduction when possible
  bool at_mmi = false;                // the launch computes a cluster's first mutated node
  bool* kill_fused = nullptr;
};

mure_status timing_begin(mure_ctx* ctx) {
  while (ctx->tevents.size() < ctx->tevents_used + 2) {
    hipEvent_t ev;
    hipError_t ee = hipEventCreate(&ev);
    if (ee != hipSuccess) return ctx->dev_fail(ee, "hipEventCreate");
    ctx->tevents.push_back(ev);
  }
  hipError_t ee = hipEventRecord(ctx->tevents[ctx->tevents_used], ctx->stream);
  if (ee != hipSuccess) return ctx->dev_fail(ee, "hipEventRecord");
  return MURE_OK;
}

// Launch node v over rows of slots [slot0, slot0 + nslots) of a chunk with
// nx inputs starting at x0.
mure_status exec_node(mure_ctx* ctx, int v, const std::vector<Where>& ins, void* out, int out_mode,
                      const void* const* wtab, const float* const* btab, int slot0, int nslots,
                      int nx, int x0, int64_t chunk_rows, int64_t alg_macs = 0, bool timed = false,
                      const Extra& ex = Extra()) {
  const Graph& g = ctx->g;
  const Node& n = g.nodes[v];
  const int out_f32 = v == g.out() ? 1 : 0;
  hipError_t e = hipSuccess;
  if (n.weighted()) {
    const int fam = node_family(g, v);
    timed = timed && ctx->kernel_timing;
    if (timed) {
      mure_status st = timing_begin(ctx);
      if (st != MURE_OK) return st;
    }
    int64_t exec_macs = ex.exec_macs >= 0 ? ex.exec_macs : (int64_t)nslots * nx * n.macs;
    if (fam == FAM_DENSE) {
      DenseArgs a;
      a.in.p = ins[0].p; a.in.mode = ins[0].mode; a.in.row_elems = n.c_in;
      a.out = out; a.out_mode = out_mode; a.out_f32 = out_f32;
      a.wtab = wtab; a.btab = btab;
      a.slot0 = slot0; a.nx = nx; a.x0 = x0; a.K = n.c_in; a.Cout = n.c_out; a.relu = n.relu;
      if (ex.vin) a.vin = *ex.vin;
      if (ex.cols) {
        a.cols = ex.cols; a.ncols = ex.ncols; a.col_slot0 = ex.col_slot0; a.delta_T = ex.delta_T;
      }
      if (ex.kill && !ex.cols && n.c_out <= 64 && out_mode == MODE_BUF) {
        const KillArgs& k = *ex.kill;
        a.do_kill = 1;
        a.write_out = 0;
        a.slot_mutant = k.slot_mutant; a.label = k.label; a.orig_ok = k.orig_ok;
        a.kill_words = k.kill_words; a.nwords = k.nwords; a.nonfinite = k.nonfinite;
        a.logits_out = k.logits_out;
        if (ex.kill_fused) *ex.kill_fused = true;
      }
      e = launch_dense(a, nslots, g.dtype, ctx->stream);
    } else if (fam == FAM_EMBED || fam == FAM_LSTM) {
      if (ex.vin || ex.cols || ex.ch_off) return ctx->fail(MURE_E_INVALID, "internal: delta or virtual input to a sequence layer");
      SeqArgs a;
      a.in.p = ins[0].p; a.in.mode = ins[0].mode; a.in.row_elems = (int64_t)n.inH * n.inW * n.inC;
      a.out = out; a.out_mode = out_mode; a.out_f32 = out_f32; a.out_row = n.out_elems();
      a.wtab = wtab;
      a.slot0 = slot0; a.nslots = nslots; a.nx = nx; a.x0 = x0;
      a.T = n.inW; a.D = fam == FAM_EMBED ? n.c_out : n.c_in; a.H = n.c_out; a.V = n.c_in; a.seq = n.seq;
      e = fam == FAM_EMBED ? launch_embed(a, ctx->stream) : launch_lstm(a, ctx->stream);
    } else if (fam == FAM_DW) {
      DwArgs a;
      a.in.p = ins[0].p; a.in.mode = ins[0].mode; a.in.row_elems = (int64_t)n.inH * n.inW * n.inC;
      a.out = out; a.out_mode = out_mode; a.out_f32 = out_f32; a.out_row = n.out_elems();
      a.wtab = wtab; a.btab = btab;
      a.slot0 = slot0; a.nslots = nslots; a.nx = nx; a.x0 = x0;
      a.H = n.inH; a.W = n.inW; a.C = n.C; a.Ho = n.H; a.Wo = n.W;
      a.kh = n.kh; a.kw = n.kw; a.stride = n.stride; a.pad = n.pad; a.relu = n.relu;
      a.ch_off = ex.ch_off; a.ch_list = ex.ch_list;
      if (ex.delta_T > 0) { a.delta_T = ex.delta_T; a.out_row = (int64_t)n.H * n.W * ex.delta_T; }
      if (ex.vin || ex.cols) return ctx->fail(MURE_E_INVALID, "internal: virtual input or columns to a depthwise convolution");
      e = launch_dw(a, g.dtype, ctx->stream);
    } else if (fam == FAM_VALU) {
      ValuArgs a;
      a.in.p = ins[0].p; a.in.mode = ins[0].mode; a.in.row_elems = (int64_t)n.inH * n.inW * n.inC;
      a.out = out; a.out_mode = out_mode; a.out_f32 = out_f32; a.out_row = n.out_elems();
      a.wtab = wtab; a.btab = btab;
      a.slot0 = slot0; a.nslots = nslots; a.nx = nx; a.x0 = x0;
      a.H = n.inH; a.W = n.inW; a.C = n.inC; a.Hp = n.H; a.Wp = n.W;
      a.Cout = n.c_out; a.kh = n.kh; a.kw = n.kw; a.stride = n.stride; a.pad = n.pad;
      a.relu = n.relu; a.pool = n.maxpool ? 1 : 0; a.K = (int)n.fan_in;
      a.ch_off = ex.ch_off; a.ch_list = ex.ch_list;
      if (ex.delta_T > 0) { a.delta_T = ex.delta_T; a.out_row = (int64_t)n.H * n.W * ex.delta_T; }
      if (ex.vin) return ctx->fail(MURE_E_INVALID, "internal: virtual input to a VALU convolution");

      e = launch_valu(a, g.dtype, ctx->stream);
    } else {
      ConvArgs a;
      a.in.p = ins[0].p;
      a.in.mode = ins[0].mode;
      a.in.row_elems = (int64_t)n.inH * n.inW * n.inC;
      a.out = out;
      a.out_mode = out_mode;
      a.out_row = n.out_elems();
      a.out_f32 = out_f32;
      a.wtab = wtab;
      a.btab = btab;
      a.slot0 = slot0;
      a.nx = nx;
      a.x0 = x0;
      if (n.kind == K_CONV) {
        a.H = n.inH; a.W = n.inW; a.C = n.inC;
        a.Hc = n.Hc; a.Wc = n.Wc; a.Hp = n.H; a.Wp = n.W;
        a.kh = n.kh; a.kw = n.kw; a.stride = n.stride; a.pad = n.pad; a.pool = n.maxpool ? 1 : 0;
      } else {
        a.H = 1; a.W = 1; a.C = n.c_in;
        a.Hc = a.Wc = a.Hp = a.Wp = 1;
        a.kh = a.kw = a.stride = 1; a.pad = 0; a.pool = 0;
      }
      a.Cout = n.c_out;
      a.relu = n.relu;
      a.K = a.kh * a.kw * a.C;
      a.P = a.pool ? 4 * a.Hp * a.Wp : a.Hc * a.Wc;
      a.tile = (int)ctx->conv_tile;
      if (ex.cols) {
        if (fam != FAM_LDS && fam != FAM_BIG && fam != FAM_GEMM && fam != FAM_HALO)
          return ctx->fail(MURE_E_INVALID, "internal: gathered delta on a kernel without columns");
        a.cols = ex.cols; a.ncols = ex.ncols; a.col_slot0 = ex.col_slot0; a.delta_T = ex.delta_T;
        if (ex.delta_T > 0) a.out_row = (int64_t)n.H * n.W * ex.delta_T;
      }
      if (ex.vin) {
        if (fam != FAM_LDS) return ctx->fail(MURE_E_INVALID, "internal: virtual input to an im2col convolution");
        a.vin = *ex.vin;
      }
      if (ex.gin || ex.gskip) {
        if (fam != FAM_HALO) return ctx->fail(MURE_E_INVALID, "internal: channel-group read by a non-halo kernel");
        if (ex.gin) a.gin = *ex.gin;
        if (ex.gskip) a.gskip = *ex.gskip;
      }
      if (ex.fuse_add >= 0) {
        const Node& an = g.nodes[ex.fuse_add];
        const Node& sn = g.nodes[an.in[1]];
        a.add_mode = an.shortcut == 1 ? 2 : 1;
        a.add_relu = an.relu;
        a.add_out_f32 = ex.fuse_add == g.out() ? 1 : 0;
        a.skip.p = ex.skip.p; a.skip.mode = ex.skip.mode; a.skip.row_elems = sn.out_elems();
        a.Hs = sn.H; a.Ws = sn.W; a.Cs = sn.C;
      }
      e = fam == FAM_LDS ? launch_conv_lds(a, nslots, ctx->stream)
        : fam == FAM_BIG ? launch_conv_big(a, nslots, ctx->stream)
        : fam == FAM_HALO ? launch_conv_halo(a, nslots, ctx->stream)
        : launch_conv(a, nslots, g.dtype, ctx->stream);
    }
    if (timed && e == hipSuccess) {
      hipError_t ee = hipEventRecord(ctx->tevents[ctx->tevents_used + 1], ctx->stream);
      if (ee != hipSuccess) return ctx->dev_fail(ee, "hipEventRecord");
      ctx->tevents_used += 2;
      ctx->tevent_family.push_back(fam);
      ctx->tevent_mmi.push_back(ex.at_mmi ? 1 : 0);
      ctx->stats.gemm_launches++;
      ctx->stats.gemm_macs_algorithmic += alg_macs;
      ctx->stats.gemm_macs_executed += exec_macs;
      ctx->stats.kernel_launches[fam]++;
      ctx->stats.kernel_macs_algorithmic[fam] += alg_macs;
      // algorithmic HBM bytes: each input row read once (a prefix-cache
      // tensor once for all slots), each output element written once, each
      // slot's (or column's) weights read once
      const int64_t es = g.dtype == DT_F32 ? 4 : 2;
      const int64_t in_row = (int64_t)n.inH * n.inW * n.inC * es;
      const int64_t out_ch = (int64_t)n.H * n.W * (out_f32 ? 4 : es);       // one channel of a row
      const int64_t w_row = n.fan_in * es;                                  // one neuron's weights
      int64_t bytes;
      const bool shared_in = (ins[0].mode == MODE_CACHE && !ex.vin) || ex.gin;
      if (ex.cols) {
        bytes = nx * in_row + (int64_t)ex.ncols * (nx * out_ch + w_row);
      } else if (ex.ch_off) {
        const int64_t ch = ex.delta_channels >= 0 ? ex.delta_channels : (int64_t)nslots * n.c_out;
        bytes = nx * in_row + ch * (nx * out_ch + w_row);
      } else {
        bytes = (shared_in ? nx : (int64_t)nslots * nx) * in_row +
                (int64_t)nslots * nx * n.c_out * out_ch + (int64_t)nslots * n.c_out * w_row;
        if (ex.fuse_add >= 0) {
          const int64_t skip_row = g.nodes[g.nodes[ex.fuse_add].in[1]].out_elems() * es;
          bytes += (ex.skip.mode == MODE_CACHE || ex.gskip ? nx : (int64_t)nslots * nx) * skip_row;
        }
      }
      ctx->stats.kernel_bytes_algorithmic[fam] += (double)bytes;
    }
  } else if (n.kind == K_ADD) {
    const Node& s = g.nodes[n.in[1]];
    AddArgs a;
    a.a.p = ins[0].p; a.a.mode = ins[0].mode; a.a.row_elems = n.out_elems();
    a.s.p = ins[1].p; a.s.mode = ins[1].mode; a.s.row_elems = s.out_elems();
    a.out = out; a.out_mode = out_mode; a.out_f32 = out_f32;
    a.nx = nx; a.x0 = x0; a.rows = chunk_rows;
    a.H = n.H; a.W = n.W; a.C = n.C; a.Hs = s.H; a.Ws = s.W; a.Cs = s.C;
    a.shortcut = n.shortcut; a.relu = n.relu;
    e = launch_add(a, g.dtype, ctx->stream);
  } else if (n.kind == K_GAP) {
    GapArgs a;
    a.in.p = ins[0].p; a.in.mode = ins[0].mode; a.in.row_elems = (int64_t)n.inH * n.inW * n.inC;
    a.out = out; a.out_mode = out_mode; a.out_f32 = out_f32;
    a.nx = nx; a.x0 = x0; a.rows = chunk_rows; a.P = n.inH * n.inW; a.C = n.C;
    e = launch_gap(a, g.dtype, ctx->stream);
  } else if (n.kind == K_FLATTEN) {
    // a view: the rows are copied; a cached output (run_original, one slot)
    // takes the chunk's rows from input x0 on
    TensorArg src;
    src.p = ins[0].p; src.mode = ins[0].mode; src.row_elems = n.out_elems();
    const int es = (int)esize_of(g, n.in[0]);
    char* dst = static_cast<char*>(out);
    if (out_mode == MODE_CACHE) {
      if (chunk_rows != nx) return ctx->fail(MURE_E_INVALID, "internal: cached FLATTEN over several slots");
      dst += (int64_t)x0 * n.out_elems() * es;
    }
    e = launch_copy_rows(src, dst, chunk_rows, nx, x0, es, ctx->stream);
  } else {
    return ctx->fail(MURE_E_INVALID, "node without a layer function");
  }
  if (e != hipSuccess) return ctx->dev_fail(e, "kernel launch");
  ctx->stats.launches++;
  return MURE_OK;
}

// Invalidate the prefix cache; its device buffers stay allocated for reuse.
void reset_cache(mure_ctx* ctx) { ctx->N = 0; }

}  // namespace

// =========================================================================
extern "C" {

int32_t mure_version(void) { return MURE_VERSION; }

static mure_status create_impl(mure_ctx** out, int32_t device, void* hip_stream) {
  if (!out) {
    g_create_error = "out is NULL";
    return MURE_E_INVALID;
  }
  *out = nullptr;
  std::unique_ptr<mure_ctx> ctx(new mure_ctx());
  if (device < 0) {
    if (device != -1) { g_create_error = "device must be >= 0, or -1 for a planning-only context"; return MURE_E_INVALID; }
    ctx->plan_only = true;
  } else {
    int count = 0;
    hipError_t e = hipGetDeviceCount(&count);
    if (e != hipSuccess) { g_create_error = std::string("hipGetDeviceCount: ") + hipGetErrorString(e); return MURE_E_DEVICE; }
    if (device >= count) { g_create_error = "no such device"; return MURE_E_INVALID; }
    e = hipSetDevice(device);
    if (e != hipSuccess) { g_create_error = std::string("hipSetDevice: ") + hipGetErrorString(e); return MURE_E_DEVICE; }
    ctx->device = device;
    ctx->stream = reinterpret_cast<hipStream_t>(hip_stream);
    e = noalloc_scratch(device, &ctx->scratch);
    if (e != hipSuccess) { g_create_error = std::string("scratch address: ") + hipGetErrorString(e); return MURE_E_DEVICE; }
    if (hipEventCreate(&ctx->ev0) != hipSuccess || hipEventCreate(&ctx->ev1) != hipSuccess) {
      g_create_error = "hipEventCreate failed";
      return MURE_E_DEVICE;
    }
  }
  *out = ctx.release();
  return MURE_OK;
}

static void destroy_impl(mure_ctx* ctx) {
  if (!ctx) return;
  if (!ctx->plan_only) {
    (void)hipSetDevice(ctx->device);
    (void)hipStreamSynchronize(ctx->stream);
    if (ctx->ev0) (void)hipEventDestroy(ctx->ev0);
    if (ctx->ev1) (void)hipEventDestroy(ctx->ev1);
    for (hipEvent_t e : ctx->tevents) (void)hipEventDestroy(e);
  }
  delete ctx;
}

const char* mure_last_error(const mure_ctx* ctx) {
  if (!ctx) return g_create_error.c_str();
  return ctx->err.c_str();
}

static mure_status set_option_impl(mure_ctx* ctx, const char* name, int64_t value) {
  if (!ctx || !name) return MURE_E_INVALID;
  const std::string n(name);
  if (n == "max_workspace_mb") {
    if (value < 1) return ctx->fail(MURE_E_INVALID, "max_workspace_mb must be >= 1");
    ctx->max_ws_mb = value;
  } else if (n == "max_device_mb") {
    if (value < 0) return ctx->fail(MURE_E_INVALID, "max_device_mb must be >= 0");
    ctx->max_device_mb = value;
  } else if (n == "chunk_inputs") {
    if (value < 0 || value % 64) return ctx->fail(MURE_E_INVALID, "chunk_inputs must be 0 or a multiple of 64");
    ctx->chunk_inputs = value;
  } else if (n == "fused_paths") {
    if (value != 0 && value != 1) return ctx->fail(MURE_E_INVALID, "fused_paths must be 0 or 1");
    ctx->fused = value;
  } else if (n == "vanilla") {
    if (value != 0 && value != 1) return ctx->fail(MURE_E_INVALID, "vanilla must be 0 or 1");
    ctx->vanilla = value;
  } else if (n == "conv_tile") {
    if (value < 0 || value > 2) return ctx->fail(MURE_E_INVALID, "conv_tile must be 0, 1 or 2");
    ctx->conv_tile = value;
  } else if (n == "group_reads") {
    if (value != 0 && value != 1) return ctx->fail(MURE_E_INVALID, "group_reads must be 0 or 1");
    ctx->group_reads = value;
  } else if (n == "kernel_timing") {
    if (value != 0 && value != 1) return ctx->fail(MURE_E_INVALID, "kernel_timing must be 0 or 1");
    ctx->kernel_timing = value;
  } else {
    return ctx->fail(MURE_E_INVALID, "unknown option " + n);
  }
  return MURE_OK;
}

static mure_status load_model_impl(mure_ctx* ctx, const mure_layer* layers, int32_t n_layers,
                            const int32_t in_hwc[3], int32_t dtype, const void* const* weights,
                            const float* const* biases) {
  if (!ctx) return MURE_E_INVALID;
  if (!layers || !in_hwc || n_layers < 2) return ctx->fail(MURE_E_INVALID, "layers/in_hwc missing or fewer than 2 nodes");
  Graph g;
  g.nodes.resize(n_layers);
  for (int i = 0; i < n_layers; ++i) {
    const mure_layer& L = layers[i];
    Node& v = g.nodes[i];
    v.kind = L.kind; v.n_in = L.n_in; v.in[0] = L.in[0]; v.in[1] = L.in[1];
    v.c_in = L.c_in; v.c_out = L.c_out; v.kh = L.kh; v.kw = L.kw; v.stride = L.stride; v.pad = L.pad;
    v.relu = L.relu; v.maxpool = L.maxpool; v.shortcut = L.shortcut; v.seq = L.seq;
    if (v.kind == K_ADD || v.kind == K_GAP || v.kind == K_FLATTEN || v.kind == K_INPUT) {
      if (v.kh > 1 || v.kw > 1) return ctx->fail(MURE_E_INVALID, "geometry given for a node without weights");
    }
  }
  std::string m = build_graph(g, in_hwc[0], in_hwc[1], in_hwc[2], dtype);
  if (!m.empty()) return ctx->fail(MURE_E_INVALID, m);
  for (int i = 0; i < n_layers; ++i) {
    const bool need = g.nodes[i].weighted();
    const bool hw = weights && weights[i], hb = biases && biases[i];
    if (need && (!hw || !hb)) return ctx->fail(MURE_E_INVALID, "node " + std::to_string(i) + ": weights and bias required");
    if (!need && (hw || hb)) return ctx->fail(MURE_E_INVALID, "node " + std::to_string(i) + ": has no parameters");
  }
  if (!ctx->plan_only) {
    HIPTRY(hipSetDevice(ctx->device));
    // from here on a device failure leaves the context without a model
    ctx->state = 0;
    ctx->have_graph = false;
    const int64_t es = dtype == DT_F32 ? 4 : 2;
    while ((int)ctx->d_w.size() < n_layers) {
      ctx->d_w.emplace_back(new DevBuf());
      ctx->d_b.emplace_back(new DevBuf());
    }
    for (int i = 0; i < n_layers; ++i) {
      if (!g.nodes[i].weighted()) continue;
      const size_t wb = (size_t)g.nodes[i].n_weights() * es, bb = (size_t)g.nodes[i].c_out * 4;
      HIPTRY(ctx->d_w[i]->ensure(wb));
      HIPTRY(ctx->d_b[i]->ensure(bb));
      if (g.nodes[i].kind == K_EMBED) {
        // token-major on the device ([V][D]): a token's D values are one
        // contiguous row for the gather
        const Node& e = g.nodes[i];
        std::vector<unsigned char> t(wb);
        const unsigned char* src = static_cast<const unsigned char*>(weights[i]);
        for (int64_t d = 0; d < e.c_out; ++d)
          for (int64_t v = 0; v < e.c_in; ++v)
            std::memcpy(&t[(size_t)((v * e.c_out + d) * es)], src + (size_t)((d * e.c_in + v) * es), (size_t)es);
        HIPTRY(hipMemcpyAsync(ctx->d_w[i]->p, t.data(), wb, hipMemcpyHostToDevice, ctx->stream));
        HIPTRY(hipStreamSynchronize(ctx->stream));
      } else if (node_family(g, i) == FAM_HALO) {
        // chunk-major for the halo kernel (bf16): KRSC weight (n, tap, ci)
        // moves to halo_w_index(n, tap, ci, C_out)
        const Node& cv = g.nodes[i];
        std::vector<uint16_t> t((size_t)cv.n_weights());
        const uint16_t* src = static_cast<const uint16_t*>(weights[i]);
        for (int n = 0; n < cv.c_out; ++n)
          for (int tap = 0; tap < 9; ++tap)
            for (int ci = 0; ci < cv.inC; ++ci)
              t[(size_t)halo_w_index(n, tap, ci, cv.c_out)] = src[((size_t)n * 9 + tap) * cv.inC + ci];
        HIPTRY(hipMemcpyAsync(ctx->d_w[i]->p, t.data(), wb, hipMemcpyHostToDevice, ctx->stream));
        HIPTRY(hipStreamSynchronize(ctx->stream));
      } else {
        HIPTRY(hipMemcpyAsync(ctx->d_w[i]->p, weights[i], wb, hipMemcpyHostToDevice, ctx->stream));
      }
      HIPTRY(hipMemcpyAsync(ctx->d_b[i]->p, biases[i], bb, hipMemcpyHostToDevice, ctx->stream));
    }
    HIPTRY(hipStreamSynchronize(ctx->stream));
  }
  ctx->g = std::move(g);
  ctx->have_graph = true;
  ctx->plan = Plan();
  ctx->recs.clear();
  reset_cache(ctx);
  ctx->stats = mure_stats{};
  ctx->state = 1;
  return MURE_OK;
}

// A run of n 4-byte values at pool offset off, copied from src (zeros where
// src is null).
struct PoolSeg {
  const void* src;
  int64_t off, n;
};

// Fill the pool from its runs; a pool of 64 MB or more (GF noise is fan-in
// long per record: 300 MB on resnet18w) is copied by up to 8 threads, each
// taking a contiguous range of runs of about equal bytes.
static void fill_pool(float* dst, const std::vector<PoolSeg>& segs, int64_t pool_n) {
  auto run = [&](size_t a, size_t b) {
    for (size_t i = a; i < b; ++i) {
      const PoolSeg& q = segs[i];
      if (q.src) std::memcpy(dst + q.off, q.src, (size_t)q.n * 4);
      else std::memset(dst + q.off, 0, (size_t)q.n * 4);
    }
  };
  const unsigned hw = std::max(1u, std::thread::hardware_concurrency());
  const int nt = pool_n * 4 >= (int64_t(64) << 20) ? (int)std::min(8u, hw) : 1;
  if (nt <= 1 || segs.size() < 2) {
    run(0, segs.size());
    return;
  }
  const int64_t per = pool_n / nt + 1;
  std::vector<std::thread> th;
  size_t i0 = 0;
  int64_t acc = 0;
  for (size_t i = 0; i < segs.size() && (int)th.size() + 1 < nt; ++i) {
    acc += segs[i].n;
    if (acc >= per) {
      th.emplace_back(run, i0, i + 1);
      i0 = i + 1;
      acc = 0;
    }
  }
  run(i0, segs.size());
  for (auto& t : th) t.join();
}

static mure_status apply_mutants_impl(mure_ctx* ctx, int32_t n_mutants, const mure_record* records,
                               int64_t n_records) {
  if (!ctx) return MURE_E_INVALID;
  if (ctx->state < 1) return ctx->fail(MURE_E_STATE, "load_model first");
  if (n_mutants < 0 || n_records < 0 || (n_records > 0 && !records))
    return ctx->fail(MURE_E_INVALID, "bad mutant/record counts");
  const Graph& g = ctx->g;
  std::vector<Record> recs(n_records);
  // the per-record float pool (GF noise; WS permutation bits, then its
  // scratch), copied straight from the callers' arrays into the staging block
  std::vector<PoolSeg> segs;
  int64_t pool_n = 0;
  for (int64_t r = 0; r < n_records; ++r) {
    const mure_record& x = records[r];
    Record& y = recs[r];
    y.mutant = x.mutant; y.op = x.op; y.layer = x.layer; y.neuron = x.neuron; y.partner = x.partner;
    y.noise_off = 0; y.noise_len = 0;
    if (x.op == OP_GF) {
      if (!x.noise || x.noise_len <= 0)
        return ctx->fail(MURE_E_INVALID, "record " + std::to_string(r) + ": Gaussian fuzz needs noise");
      y.noise_off = pool_n;
      y.noise_len = x.noise_len;
      if (x.layer >= 0 && x.layer < (int)g.nodes.size() && x.noise_len == g.nodes[x.layer].fan_in) {
        segs.push_back(PoolSeg{x.noise, pool_n, x.noise_len});
        pool_n += x.noise_len;
      }
    } else if (x.op == OP_WS) {
      if (!x.perm || x.noise_len <= 0)
        return ctx->fail(MURE_E_INVALID, "record " + std::to_string(r) + ": weight shuffle needs a permutation");
      y.noise_len = x.noise_len;
      if (x.layer >= 0 && x.layer < (int)g.nodes.size() && x.noise_len == g.nodes[x.layer].fan_in) {
        std::vector<char> seen((size_t)x.noise_len, 0);
        for (int64_t k = 0; k < x.noise_len; ++k) {
          const int32_t q = x.perm[k];
          if (q < 0 || q >= x.noise_len || seen[q])
            return ctx->fail(MURE_E_INVALID, "record " + std::to_string(r) + ": perm is not a permutation");
          seen[q] = 1;
        }
        y.noise_off = pool_n;                              // 4-byte integers in the float pool
        segs.push_back(PoolSeg{x.perm, pool_n, x.noise_len});
        pool_n += x.noise_len;
        y.scratch_off = pool_n;
        segs.push_back(PoolSeg{nullptr, pool_n, x.noise_len});
        pool_n += x.noise_len;
      }
    }
  }
  Plan plan;
  std::string m = build_plan(g, n_mutants, recs, plan, ctx->vanilla != 0);
  if (!m.empty()) return ctx->fail(MURE_E_INVALID, m);

  // copy-on-write pool: weights (256-byte aligned) then biases
  const int64_t es = g.dtype == DT_F32 ? 4 : 2;
  std::vector<int64_t> woff(plan.cows.size()), boff(plan.cows.size());
  int64_t pos = 0;
  for (size_t c = 0; c < plan.cows.size(); ++c) {
    woff[c] = pos;
    pos += (g.nodes[plan.cows[c].layer].n_weights() * es + 255) / 256 * 256;
  }
  for (size_t c = 0; c < plan.cows.size(); ++c) {
    boff[c] = pos;
    pos += ((int64_t)g.nodes[plan.cows[c].layer].c_out * 4 + 255) / 256 * 256;
  }
  if (ctx->max_device_mb > 0 && model_bytes(g) + pos > (ctx->max_device_mb << 20))
    return ctx->fail(MURE_E_NOMEM, "the model and the mutants' copy-on-write layers need " +
                                       std::to_string((model_bytes(g) + pos) >> 20) + " MB, above max_device_mb = " +
                                       std::to_string(ctx->max_device_mb));
  ctx->cow_bytes = pos;

  if (!ctx->plan_only) {
    HIPTRY(hipSetDevice(ctx->device));
    HIPTRY(hipEventRecord(ctx->ev0, ctx->stream));
    // from here on a device failure leaves the context without mutants
    ctx->state = 1;
    ctx->plan = Plan();
    HIPTRY(ctx->d_cow.ensure((size_t)std::max<int64_t>(pos, 256)));
    char* base = ctx->d_cow.as<char>();
    std::map<std::pair<int, int>, size_t> cow_index;
    std::vector<CowArgs> cargs(plan.cows.size());
    std::vector<DevRecord> drecs;
    for (size_t c = 0; c < plan.cows.size(); ++c) {
      const CowCopy& cc = plan.cows[c];
      CowArgs& a = cargs[c];
      a.w_src = ctx->d_w[cc.layer]->p;
      a.w_dst = base + woff[c];
      a.b_src = ctx->d_b[cc.layer]->as<float>();
      a.b_dst = reinterpret_cast<float*>(base + boff[c]);
      a.c_out = g.nodes[cc.layer].c_out;
      a.fan_in = g.nodes[cc.layer].fan_in;
      const bool tok_major = g.nodes[cc.layer].kind == K_EMBED;      // stored [V][D]
      a.rs = tok_major ? 1 : a.fan_in;
      a.ks = tok_major ? a.c_out : 1;
      a.halo_c = node_family(g, cc.layer) == FAM_HALO ? g.nodes[cc.layer].inC : 0;
      a.rec0 = (int)drecs.size();
      for (int r : cc.records) {
        DevRecord d;
        d.op = recs[r].op; d.neuron = recs[r].neuron; d.partner = recs[r].partner; d.pad = 0;
        d.noise_off = recs[r].noise_off;
        d.scratch_off = recs[r].scratch_off;
        drecs.push_back(d);
      }
      a.rec1 = (int)drecs.size();
      cow_index[{cc.mutant, cc.layer}] = c;
    }
    // pointer tables: per group, per weighted node >= mmi, one pointer per slot;
    // plus 1-entry tables of the original parameters (run_original)
    std::vector<const void*> tabs;
    std::vector<mure_ctx::GroupTabs> gtabs(plan.groups.size());
    std::vector<int32_t> slots, chmaps;
    std::map<int, int64_t> ow, ob;
    for (int v = 0; v < (int)g.nodes.size(); ++v) {
      if (!g.nodes[v].weighted()) continue;
      ow[v] = (int64_t)tabs.size(); tabs.push_back(ctx->d_w[v]->p);
      ob[v] = (int64_t)tabs.size(); tabs.push_back(ctx->d_b[v]->p);
    }
    for (size_t gi = 0; gi < plan.groups.size(); ++gi) {
      const Group& gr = plan.groups[gi];
      mure_ctx::GroupTabs& gt = gtabs[gi];
      for (int v = gr.mmi; v < (int)g.nodes.size(); ++v) {
        if (!g.nodes[v].weighted()) continue;
        gt.w[v] = (int64_t)tabs.size();
        for (int mu : gr.mutants) {
          auto it = cow_index.find({mu, v});
          tabs.push_back(it == cow_index.end() ? ctx->d_w[v]->p : cargs[it->second].w_dst);
        }
        gt.b[v] = (int64_t)tabs.size();
        for (int mu : gr.mutants) {
          auto it = cow_index.find({mu, v});
          tabs.push_back(it == cow_index.end() ? ctx->d_b[v]->p : (const void*)cargs[it->second].b_dst);
        }
      }
      gt.slot_mutant = (int64_t)slots.size();
      for (int mu : gr.mutants) slots.push_back(mu);
      gt.chmap = (int64_t)chmaps.size();
      for (size_t s = 0; s < gr.mutants.size(); ++s) {
        const std::vector<int>& cm = plan.mutants[gr.mutants[s]].chmap;
        chmaps.insert(chmaps.end(), cm.begin(), cm.end());
      }
      gt.vchmap = (int64_t)chmaps.size();
      chmaps.insert(chmaps.end(), gr.vchmap.begin(), gr.vchmap.end());
      // channel-group reads: a side plane per (slot, changed 8-channel group)
      gt.vgbeg.assign(1, 0);
      if (gr.vhalo) {
        const int C = g.nodes[gr.mmi].c_out, G = C / 8;
        std::vector<int32_t> src((size_t)gr.mutants.size() * G, -1), ent;
        int32_t e = 0;
        for (size_t s = 0; s < gr.mutants.size(); ++s) {
          const int* row = &gr.vchmap[s * C];
          for (int q = 0; q < G; ++q) {
            bool changed = false;
            for (int j = 0; j < 8; ++j) changed = changed || row[8 * q + j] != 8 * q + j;
            if (!changed) continue;
            src[s * G + q] = e++;
            ent.push_back((int32_t)s);
            ent.push_back(q);
          }
          gt.vgbeg.push_back(e);
        }
        gt.vgsrc = (int64_t)chmaps.size();
        chmaps.insert(chmaps.end(), src.begin(), src.end());
        gt.vgent = (int64_t)chmaps.size();
        chmaps.insert(chmaps.end(), ent.begin(), ent.end());
      }
    }
    // touched-channel lists of the recompute mutants (CSR, absolute offsets
    // into the list stored after every group's offsets)
    {
      std::vector<int32_t> offs, list;
      std::vector<int64_t> where(plan.groups.size());
      for (size_t gi = 0; gi < plan.groups.size(); ++gi) {
        const Group& gr = plan.groups[gi];
        where[gi] = (int64_t)offs.size();
        for (int s = 0; s < gr.n_recompute; ++s) {
          offs.push_back((int32_t)list.size());
          const std::vector<int>& tl = plan.mutants[gr.mutants[s]].touched_list;
          list.insert(list.end(), tl.begin(), tl.end());
        }
        offs.push_back((int32_t)list.size());
      }
      const int64_t base = (int64_t)slots.size();
      for (size_t gi = 0; gi < plan.groups.size(); ++gi) gtabs[gi].choff = base + where[gi];
      const int64_t list_base = base + (int64_t)offs.size();
      for (int32_t& o : offs) o += (int32_t)list_base;
      slots.insert(slots.end(), offs.begin(), offs.end());
      slots.insert(slots.end(), list.begin(), list.end());
    }
    // gathered delta columns of the recompute slots: (group slot, channel, t)
    std::vector<DeltaCol> cols;
    for (size_t gi = 0; gi < plan.groups.size(); ++gi) {
      const Group& gr = plan.groups[gi];
      mure_ctx::GroupTabs& gt = gtabs[gi];
      gt.cols = (int64_t)cols.size();
      gt.colbeg.assign(1, 0);
      for (int s = 0; s < gr.n_recompute; ++s) {
        const std::vector<int>& tl = plan.mutants[gr.mutants[s]].touched_list;
        for (size_t t = 0; t < tl.size(); ++t) cols.push_back(DeltaCol{s, tl[t], (int)t, 0});
        gt.colbeg.push_back((int64_t)cols.size() - gt.cols);
      }
    }
    // one upload: every table at a 256-byte aligned offset of one block
    size_t total = 0;
    auto section = [&](size_t bytes) {
      const size_t o = total;
      total += (bytes + 255) / 256 * 256;
      return o;
    };
    const size_t o_tabs = section(tabs.size() * sizeof(void*));
    const size_t o_slots = section(slots.size() * 4);
    const size_t o_chmap = section(chmaps.size() * 4);
    const size_t o_cols = section(cols.size() * sizeof(DeltaCol));
    const size_t o_cargs = section(cargs.size() * sizeof(CowArgs));
    const size_t o_drecs = section(drecs.size() * sizeof(DevRecord));
    const size_t o_noise = section((size_t)pool_n * 4);
    HIPTRY(ctx->h_apply.ensure(std::max<size_t>(total, 256)));
    HIPTRY(ctx->d_apply.ensure(std::max<size_t>(total, 256)));
    char* h = static_cast<char*>(ctx->h_apply.p);
    auto put = [&](size_t off, const void* src, size_t bytes) {
      if (bytes) std::memcpy(h + off, src, bytes);
    };
    put(o_tabs, tabs.data(), tabs.size() * sizeof(void*));
    put(o_slots, slots.data(), slots.size() * 4);
    put(o_chmap, chmaps.data(), chmaps.size() * 4);
    put(o_cols, cols.data(), cols.size() * sizeof(DeltaCol));
    put(o_cargs, cargs.data(), cargs.size() * sizeof(CowArgs));
    put(o_drecs, drecs.data(), drecs.size() * sizeof(DevRecord));
    fill_pool(reinterpret_cast<float*>(h + o_noise), segs, pool_n);
    hipStream_t st = ctx->stream;
    char* d = ctx->d_apply.as<char>();
    if (total) HIPTRY(hipMemcpyAsync(d, h, total, hipMemcpyHostToDevice, st));
    ctx->tables = reinterpret_cast<const void**>(d + o_tabs);
    ctx->slotv = reinterpret_cast<int32_t*>(d + o_slots);
    ctx->chmapv = reinterpret_cast<int32_t*>(d + o_chmap);
    ctx->colv = reinterpret_cast<DeltaCol*>(d + o_cols);
    if (!cargs.empty())
      HIPTRY(launch_cow(reinterpret_cast<const CowArgs*>(d + o_cargs), (int)cargs.size(),
                        reinterpret_cast<const DevRecord*>(d + o_drecs), reinterpret_cast<const float*>(d + o_noise),
                        g.dtype, st));
    HIPTRY(hipEventRecord(ctx->ev1, ctx->stream));
    HIPTRY(hipEventSynchronize(ctx->ev1));
    float ms = 0.f;
    (void)hipEventElapsedTime(&ms, ctx->ev0, ctx->ev1);
    ctx->stats.ms_apply = ms;
    ctx->gtabs = std::move(gtabs);
    ctx->orig_w = std::move(ow);
    ctx->orig_b = std::move(ob);
  }
  ctx->plan = std::move(plan);
  ctx->recs = std::move(recs);
  reset_cache(ctx);
  ctx->stats.n_groups = (int64_t)ctx->plan.groups.size();
  ctx->stats.n_identity_mutants = ctx->plan.n_identity;
  ctx->state = 2;
  return MURE_OK;
}


// -------------------------------------------------------------------------
// run_original: the original model once over X; fills the prefix cache.
static mure_status run_original_impl(mure_ctx* ctx, const void* inputs_dev, int64_t n_inputs,
                              const int32_t* labels) {
  if (!ctx) return MURE_E_INVALID;
  if (ctx->plan_only) return ctx->fail(MURE_E_UNSUPPORTED, "planning-only context");
  if (ctx->state < 2) return ctx->fail(MURE_E_STATE, "apply_mutants must run before run_original");
  if (!inputs_dev || n_inputs < 1 || n_inputs > (int64_t)1 << 30)
    return ctx->fail(MURE_E_INVALID, "inputs missing or n_inputs out of range");
  const Graph& g = ctx->g;
  const int C = g.classes();
  const int L = g.out();
  if (labels)
    for (int64_t i = 0; i < n_inputs; ++i)
      if (labels[i] < 0 || labels[i] >= C) return ctx->fail(MURE_E_INVALID, "label out of range");
  const int64_t n = n_inputs;
  std::set<int> cached(ctx->plan.cache_nodes.begin(), ctx->plan.cache_nodes.end());
  if (ctx->max_device_mb > 0) {
    int64_t need = model_bytes(g) + ctx->cow_bytes + n * C * 4;
    for (int v : cached)
      if (v != L) need += n * g.act_bytes(v);
    if (need > (ctx->max_device_mb << 20))
      return ctx->fail(MURE_E_NOMEM, "the model, the copies and the prefix cache need " + std::to_string(need >> 20) +
                                         " MB, above max_device_mb = " + std::to_string(ctx->max_device_mb));
  }
  HIPTRY(hipSetDevice(ctx->device));
  reset_cache(ctx);
  ctx->state = 2;
  int64_t cache_bytes = 0;
  for (auto it = ctx->cache.begin(); it != ctx->cache.end();)     // drop tensors no longer cached
    it = cached.count(it->first) ? std::next(it) : ctx->cache.erase(it);
  for (int v : cached) {
    if (v == L) continue;                               // the logits buffer serves the output
    auto& b = ctx->cache[v];
    if (!b) b.reset(new DevBuf());
    HIPTRY(b->ensure((size_t)(n * g.act_bytes(v))));
    cache_bytes += n * g.act_bytes(v);
  }
  HIPTRY(ctx->d_logits.ensure((size_t)(n * C * 4)));
  HIPTRY(ctx->d_label.ensure((size_t)(n * 4)));
  HIPTRY(ctx->d_ok.ensure((size_t)n));
  HIPTRY(ctx->d_classmask.ensure(64));
  HIPTRY(ctx->d_nonfinite.ensure(8));
  cache_bytes += n * C * 4;
  DevBuf& d_given = ctx->d_given;
  if (labels) {
    HIPTRY(d_given.ensure((size_t)(n * 4)));
    HIPTRY(hipMemcpyAsync(d_given.p, labels, (size_t)(n * 4), hipMemcpyHostToDevice, ctx->stream));
  }
  std::vector<int> nodes;
  for (int v = 1; v <= L; ++v) nodes.push_back(v);
  std::set<int> external(cached);
  external.insert(L);
  std::map<int, int> fused;                            // conv_b -> ADD run as one launch
  for (int v = 1; v <= L; ++v) {
    const int fa = ctx->fused ? fused_add_of(g, v) : -1;
    if (fa >= 0 && !cached.count(v)) fused[v] = fa;
  }
  Placement pl = place_buffers(g, nodes, external, fused);
  const int64_t budget = ctx->max_ws_mb << 20;
  int64_t nx = n;
  if (ctx->chunk_inputs) nx = std::min<int64_t>(nx, ctx->chunk_inputs);
  if (pl.peak * nx > budget) nx = std::max<int64_t>(64, budget / std::max<int64_t>(pl.peak, 1) / 64 * 64);
  if (nx > n) nx = n;
  HIPTRY(ctx->d_ws.ensure((size_t)(pl.peak * nx)));
  char* ws = ctx->d_ws.as<char>();

  HIPTRY(hipEventRecord(ctx->ev0, ctx->stream));
  HIPTRY(hipMemsetAsync(ctx->d_classmask.p, 0, 64, ctx->stream));
  HIPTRY(hipMemsetAsync(ctx->d_nonfinite.p, 0, 8, ctx->stream));
  if (cached.count(0))
    HIPTRY(hipMemcpyAsync(ctx->cache[0]->p, inputs_dev, (size_t)(n * g.act_bytes(0)),
                          hipMemcpyDeviceToDevice, ctx->stream));
  const void* const* tabs = ctx->tables;
  ctx->stats.launches = 0;
  for (int64_t x0 = 0; x0 < n; x0 += nx) {
    const int cnt = (int)std::min<int64_t>(nx, n - x0);
    auto where = [&](int p) -> Where {
      if (p == 0) return {cached.count(0) ? ctx->cache[0]->p : inputs_dev, MODE_CACHE};
      if (p == L) return {ctx->d_logits.p, MODE_CACHE};
      if (cached.count(p)) return {ctx->cache[p]->p, MODE_CACHE};
      return {ws + pl.offset.at(p) * nx, MODE_BUF};
    };
    std::set<int> done;
    for (int v = 1; v <= L; ++v) {
      if (done.count(v)) continue;
      const Node& nd = g.nodes[v];
      std::vector<Where> ins;
      for (int k = 0; k < nd.n_in; ++k) ins.push_back(where(nd.in[k]));
      Extra ex;
      int tgt = v;
      auto f = fused.find(v);
      if (f != fused.end()) {
        tgt = f->second;
        ex.fuse_add = tgt;
        ex.skip = where(g.nodes[tgt].in[1]);
        done.insert(tgt);
      }
      Where o = where(tgt);
      const void* const* wt = nd.weighted() ? tabs + ctx->orig_w.at(v) : nullptr;
      const float* const* bt = nd.weighted() ? reinterpret_cast<const float* const*>(tabs + ctx->orig_b.at(v)) : nullptr;
      mure_status st = exec_node(ctx, v, ins, const_cast<void*>(o.p), o.mode, wt, bt, 0, 1, cnt, (int)x0, cnt,
                                 0, false, ex);
      if (st != MURE_OK) return st;
    }
  }
  LabelArgs la;
  la.logits = ctx->d_logits.as<float>();
  la.N = n;
  la.C = C;
  la.given = labels ? d_given.as<int32_t>() : nullptr;
  la.label = ctx->d_label.as<int32_t>();
  la.ok = ctx->d_ok.as<uint8_t>();
  la.class_mask = ctx->d_classmask.as<unsigned long long>();
  la.nonfinite = ctx->d_nonfinite.as<unsigned long long>();
  HIPTRY(launch_labels(la, ctx->stream));
  HIPTRY(hipEventRecord(ctx->ev1, ctx->stream));
  HIPTRY(hipEventSynchronize(ctx->ev1));
  float ms = 0.f;
  HIPTRY(hipEventElapsedTime(&ms, ctx->ev0, ctx->ev1));
  unsigned long long mask[8];
  HIPTRY(hipMemcpy(mask, ctx->d_classmask.p, 64, hipMemcpyDeviceToHost));
  ctx->n_labels = 0;
  for (int i = 0; i < 8; ++i) ctx->n_labels += __builtin_popcountll(mask[i]);
  ctx->N = n;
  ctx->stats.ms_run_original = ms;
  ctx->stats.macs_original = g.full_macs() * n;
  ctx->stats.cache_bytes = cache_bytes;
  ctx->state = 3;
  return MURE_OK;
}

// -------------------------------------------------------------------------
// Chunking of group gi's suffix: per-row buffer placement, inputs per chunk
// (nx) and mutant slots per chunk (spc) for a workspace budget in bytes.  The
// budget is a soft cap: the smallest chunk (one slot x min(64, N) inputs) is
// used even when it needs more (need_bytes tells).
}  // extern "C"
namespace {
struct ChunkGeom {
  Placement pl;
  std::map<int, int> fused_adds;                     // conv_b -> ADD run as one launch
  int64_t nx = 0, spc = 0, cap_rows = 0, need_bytes = 0;
};

ChunkGeom group_geometry(const mure_ctx* ctx, int gi, int nslots, int64_t budget) {
  const Graph& g = ctx->g;
  const Group& gr = ctx->plan.groups[gi];
  const int L = g.out(), mmi = gr.mmi;
  const int64_t N = ctx->N;
  ChunkGeom cg;
  std::vector<int> nodes;
  for (int v = mmi; v <= L; ++v) nodes.push_back(v);
  for (int v = mmi + 1; v <= L; ++v) {
    const int fa = ctx->fused ? fused_add_of(g, v) : -1;
    if (fa >= 0) cg.fused_adds[v] = fa;
  }
  cg.pl = place_buffers(g, nodes, {}, cg.fused_adds);
  const int64_t peak = std::max<int64_t>(cg.pl.peak, 1);
  int64_t nx = N;
  if (ctx->chunk_inputs) nx = std::min<int64_t>(nx, ctx->chunk_inputs);
  if (peak * nx > budget) nx = std::max<int64_t>(64, budget / peak / 64 * 64);
  if (nx > N) nx = N;
  int64_t spc = std::max<int64_t>(1, budget / (peak * nx));
  spc = std::min<int64_t>(spc, std::min<int64_t>(65535, std::max(nslots, 1)));
  spc = std::min<int64_t>(spc, std::max<int64_t>(1, ((int64_t)1 << 31) / nx / 64));
  cg.nx = nx;
  cg.spc = spc;
  cg.cap_rows = spc * nx;
  cg.need_bytes = cg.pl.peak * cg.cap_rows;
  return cg;
}
}  // namespace
extern "C" {

// The suffix of group gi for its slots [s_begin, s_end), over all inputs.
// ws == nullptr: the context's workspace, grown as needed; otherwise ws holds
// ws_bytes and the chunks are sized to fit it (MURE_E_NOMEM if they cannot).
static mure_status run_group(mure_ctx* ctx, int gi, int s_begin, int s_end, uint64_t* kill_words,
                             float* logits_out, char* ws = nullptr, int64_t ws_bytes = 0) {
  const Graph& g = ctx->g;
  const Group& gr = ctx->plan.groups[gi];
  const mure_ctx::GroupTabs& gt = ctx->gtabs[gi];
  const int L = g.out(), mmi = gr.mmi;
  const int64_t N = ctx->N;
  int64_t budget = ctx->max_ws_mb << 20;
  if (ws) budget = std::min(budget, ws_bytes);
  const ChunkGeom cg = group_geometry(ctx, gi, s_end - s_begin, budget);
  const Placement& pl = cg.pl;
  const std::map<int, int>& fused_adds = cg.fused_adds;
  const int64_t nx = cg.nx, spc = cg.spc, cap_rows = cg.cap_rows;
  // channel-group reads of mmi's output by its halo consumers (not with a
  // caller's scratch array: the side planes live in a buffer of their own)
  const Node& nmm = g.nodes[mmi];
  const int64_t vP = (int64_t)nmm.H * nmm.W;
  const bool vh = gr.vhalo && ctx->group_reads && ctx->fused && !ws && nx * vP < INT32_MAX;
  if (vh) {
    int64_t most = 0;
    for (int cs0 = s_begin; cs0 < s_end; cs0 += (int)spc) {
      const int cs1 = (int)std::min<int64_t>(s_end, cs0 + spc);
      most = std::max<int64_t>(most, gt.vgbeg[cs1] - gt.vgbeg[cs0]);
    }
    HIPTRY(ctx->d_side.ensure((size_t)(most * nx * vP * 16)));
  }
  if (ws) {
    if (cg.need_bytes > ws_bytes) return ctx->fail(MURE_E_NOMEM, "chunk workspace exceeds the scratch array");
  } else {
    HIPTRY(ctx->d_ws.ensure((size_t)cg.need_bytes));
    ctx->stats.workspace_bytes = std::max<int64_t>(ctx->stats.workspace_bytes, (int64_t)ctx->d_ws.bytes);
    ws = ctx->d_ws.as<char>();
  }
  const void* const* tabs = ctx->tables;
  const int32_t* slot_mut = ctx->slotv + gt.slot_mutant;
  const Node& nm = g.nodes[mmi];
  const void* mmi_cache = mmi == L ? ctx->d_logits.p : (ctx->cache.count(mmi) ? ctx->cache[mmi]->p : nullptr);
  for (int cs0 = s_begin; cs0 < s_end; cs0 += (int)spc) {
    const int cs1 = (int)std::min<int64_t>(s_end, cs0 + spc);
    const int ns = cs1 - cs0;
    for (int64_t x0 = 0; x0 < N; x0 += nx) {
      const int cnt = (int)std::min<int64_t>(nx, N - x0);
      const int64_t rows = (int64_t)ns * cnt;
      auto where = [&](int p) -> Where {
        if (p < mmi) {
          if (p == 0 && !ctx->cache.count(0)) return {nullptr, MODE_CACHE};
          return {ctx->cache.at(p)->p, MODE_CACHE};
        }
        return {ws + pl.offset.at(p) * cap_rows, MODE_BUF};
      };
      KillArgs ka;
      ka.C = g.classes();
      ka.nx = cnt; ka.x0 = (int)x0; ka.nslots = ns; ka.slot0 = 0;
      ka.slot_mutant = slot_mut + cs0;
      ka.label = ctx->d_label.as<int32_t>();
      ka.orig_ok = ctx->d_ok.as<uint8_t>();
      ka.kill_words = kill_words;
      ka.nwords = (N + 63) / 64;
      ka.nonfinite = ctx->d_nonfinite.as<unsigned long long>();
      ka.logits_out = logits_out;
      bool fused = false;
      // node mmi.  Delta groups: every slot starts from the cached output
      // (patched for effect-block / switch mutants), then the touched channels
      // of the fuzz / inverse mutants are recomputed.  Otherwise the fuzz /
      // inverse mutants recompute the whole node and the others are patched.
      {
        std::vector<Where> ins;
        for (int k = 0; k < nm.n_in; ++k) ins.push_back(where(nm.in[k]));
        void* out = const_cast<void*>(where(mmi).p);
        const int rec_end = std::min(cs1, gr.n_recompute);
        const int pa = (gr.virt || vh) ? cs1 : gr.delta ? cs0 : std::max(cs0, gr.n_recompute);
        if (pa < cs1) {
          PatchArgs a;
          a.cache = mmi_cache;
          a.out = out;
          a.chmap = ctx->chmapv + gt.chmap;
          a.slot0 = pa - cs0;
          a.chmap_slot0 = pa;
          a.nx = cnt; a.x0 = (int)x0; a.nslots = cs1 - pa;
          a.P = nm.H * nm.W; a.C = nm.C; a.esize = (int)esize_of(g, mmi);
          HIPTRY(launch_patch(a, ctx->stream));
          ctx->stats.launches++;
        }
        if (cs0 < rec_end) {
          int64_t touched = 0, tl = 0;
          for (int sl = cs0; sl < rec_end; ++sl) {
            touched += ctx->plan.mutants[gr.mutants[sl]].touched;
            tl += (int64_t)ctx->plan.mutants[gr.mutants[sl]].touched_list.size();
          }
          const int64_t per_ch = nm.macs / nm.c_out;
          Extra ex;
          ex.at_mmi = true;
          int launch_slots = rec_end - cs0;
          if (gr.delta) {
            if (gr.virt || vh) ex.delta_T = gr.T;
            ex.exec_macs = tl * per_ch * cnt;
            ex.delta_channels = tl;
            if (node_family(g, mmi) == FAM_VALU || node_family(g, mmi) == FAM_DW) {
              ex.ch_off = ctx->slotv + gt.choff + cs0;
              ex.ch_list = ctx->slotv;
            } else {
              ex.cols = ctx->colv + gt.cols + gt.colbeg[cs0];
              ex.ncols = (int)(gt.colbeg[rec_end] - gt.colbeg[cs0]);
              ex.col_slot0 = cs0;
              launch_slots = ex.ncols > 0 ? 1 : 0;
            }
          }
          // the kill fuses into the output layer only when every slot of the
          // chunk is recomputed here (patched slots need the kill kernel, which
          // reads the logits buffer)
          if (mmi == L && pa >= cs1 && ctx->fused) { ex.kill = &ka; ex.kill_fused = &fused; }
          if (launch_slots > 0) {
            mure_status st = exec_node(ctx, mmi, ins, out, MODE_BUF, tabs + gt.w.at(mmi) + cs0,
                                       reinterpret_cast<const float* const*>(tabs + gt.b.at(mmi) + cs0),
                                       0, launch_slots, cnt, (int)x0, rows, touched * per_ch * cnt, true, ex);
            if (st != MURE_OK) return st;
          }
        }
      }
      // the changed 8-channel groups of every slot of the chunk, from the
      // cache, the slot's channel map and the compact delta rows
      GroupIn gin;
      if (vh) {
        const int64_t e0 = gt.vgbeg[cs0], e1 = gt.vgbeg[cs1];
        const void* cache_x0 = static_cast<const char*>(mmi_cache) + x0 * vP * nm.C * 2;
        if (e1 > e0) {
          GroupPatchArgs gpa;
          gpa.cache = cache_x0;
          gpa.chmap = ctx->chmapv + gt.vchmap;
          gpa.delta = where(mmi).p;
          gpa.ent = ctx->chmapv + gt.vgent + 2 * e0;
          gpa.side = ctx->d_side.p;
          gpa.n_ent = (int)(e1 - e0); gpa.nx = cnt; gpa.P = (int)vP; gpa.C = nm.C; gpa.T = gr.T; gpa.slot0 = cs0;
          HIPTRY(launch_group_patch(gpa, ctx->stream));
          ctx->stats.launches++;
          ctx->stats.group_planes += e1 - e0;
        }
        gin.cache = cache_x0;
        gin.src = ctx->chmapv + gt.vgsrc + (int64_t)cs0 * (nm.C / 8);
        gin.side = ctx->d_side.p;
        gin.g0 = (int)e0; gin.C = nm.C; gin.P = (int)vP;
      }
      VirtualIn vin;
      if (gr.virt) {
        vin.cache = mmi_cache;
        vin.chmap = ctx->chmapv + gt.vchmap + (int64_t)cs0 * nm.C;
        vin.delta = where(mmi).p;
        vin.C = nm.C;
        vin.HW = nm.H * nm.W;
        vin.T = gr.T;
      }
      std::set<int> done;
      for (int v = mmi + 1; v <= L; ++v) {
        if (done.count(v)) continue;
        const Node& nd = g.nodes[v];
        std::vector<Where> ins;
        for (int k = 0; k < nd.n_in; ++k) ins.push_back(where(nd.in[k]));
        auto f = fused_adds.find(v);
        if (f != fused_adds.end()) {
          const int fa = f->second;
          Extra exf;
          exf.fuse_add = fa;
          exf.skip = where(g.nodes[fa].in[1]);
          if (vh && g.nodes[fa].in[1] == mmi) exf.gskip = &gin;
          if (vh && nd.n_in == 1 && nd.in[0] == mmi) exf.gin = &gin;
          if (fa == L) { exf.kill = nullptr; }
          done.insert(fa);
          mure_status st = exec_node(ctx, v, ins, const_cast<void*>(where(fa).p), MODE_BUF,
                                     tabs + gt.w.at(v) + cs0,
                                     reinterpret_cast<const float* const*>(tabs + gt.b.at(v) + cs0), 0, ns, cnt,
                                     (int)x0, rows, rows * nd.macs, true, exf);
          if (st != MURE_OK) return st;
          continue;
        }
        const void* const* wt = nd.weighted() ? tabs + gt.w.at(v) + cs0 : nullptr;
        const float* const* bt = nd.weighted() ? reinterpret_cast<const float* const*>(tabs + gt.b.at(v) + cs0) : nullptr;
        Extra ex;
        if (v == L && ctx->fused) { ex.kill = &ka; ex.kill_fused = &fused; }
        if (vh && nd.n_in == 1 && nd.in[0] == mmi) ex.gin = &gin;
        if (gr.virt && nd.n_in == 1 && nd.in[0] == mmi) {
          // the consumer of mmi: delta groups read every slot virtually; in
          // whole-node groups the recomputed slots read their own output rows
          // and only the patched slots read the cache through their maps
          const int rec_ns = gr.delta ? 0 : std::max(0, std::min(cs1, gr.n_recompute) - cs0);
          if (rec_ns > 0) {
            Extra ex1 = ex;
            mure_status st = exec_node(ctx, v, ins, const_cast<void*>(where(v).p), MODE_BUF, wt, bt, 0, rec_ns,
                                       cnt, (int)x0, (int64_t)rec_ns * cnt, (int64_t)rec_ns * cnt * nd.macs, true, ex1);
            if (st != MURE_OK) return st;
          }
          if (rec_ns < ns) {
            ex.vin = &vin;
            mure_status st = exec_node(ctx, v, ins, const_cast<void*>(where(v).p), MODE_BUF, wt, bt, rec_ns,
                                       ns - rec_ns, cnt, (int)x0, (int64_t)(ns - rec_ns) * cnt,
                                       (int64_t)(ns - rec_ns) * cnt * nd.macs, true, ex);
            if (st != MURE_OK) return st;
          }
          continue;
        }
        mure_status st = exec_node(ctx, v, ins, const_cast<void*>(where(v).p), MODE_BUF, wt, bt, 0, ns, cnt,
                                   (int)x0, rows, rows * nd.macs, true, ex);
        if (st != MURE_OK) return st;
      }
      if (fused) continue;

      ka.logits = reinterpret_cast<const float*>(where(L).p);
      HIPTRY(launch_kill(ka, ctx->stream));
      ctx->stats.launches++;
    }
  }
  return MURE_OK;
}

}  // extern "C"

// Both run_mutants entry points.  noalloc: the kill words are the caller's,
// and the workspace, kill counts and label masks live in this GPU's scratch
// array; no device memory is allocated and no launch is timed.
static mure_status run_mutants_impl(mure_ctx* ctx, uint64_t* kill_bits_dev, int64_t* kills_host,
                                    mure_score* score, bool noalloc) {
  if (!ctx) return MURE_E_INVALID;
  if (ctx->plan_only) return ctx->fail(MURE_E_UNSUPPORTED, "planning-only context");
  if (ctx->state != 3) return ctx->fail(MURE_E_STATE, "run_original must run after the last apply_mutants");
  if (noalloc && !kill_bits_dev) return ctx->fail(MURE_E_INVALID, "kill_bits_dev is NULL");
  HIPTRY(hipSetDevice(ctx->device));
  const int64_t M = ctx->plan.n_mutants, N = ctx->N, nwords = (N + 63) / 64;
  const int C = ctx->g.classes();
  const int mw = (C + 63) / 64;
  uint64_t* kw = kill_bits_dev;
  int64_t* d_kills = nullptr;
  unsigned long long* d_masks = nullptr;
  char* ws = nullptr;
  int64_t ws_bytes = 0;
  if (noalloc) {
    // [kill counts | label masks | chunk workspace], 256-byte aligned parts
    if (!ctx->scratch) return ctx->fail(MURE_E_DEVICE, "no scratch array on this device");
    const int64_t kb = (M * 8 + 255) / 256 * 256, mb = (M * mw * 8 + 255) / 256 * 256;
    const int64_t total = (int64_t)MURE_NOALLOC_SCRATCH_BYTES;
    if (kb + mb >= total) return ctx->fail(MURE_E_NOMEM, "kill counters exceed the scratch array");
    char* base = static_cast<char*>(ctx->scratch);
    d_kills = reinterpret_cast<int64_t*>(base);
    d_masks = reinterpret_cast<unsigned long long*>(base + kb);
    ws = base + kb + mb;
    ws_bytes = total - kb - mb;
    // refuse before any device work if some cluster's smallest chunk does not fit
    for (int gi = 0; gi < (int)ctx->plan.groups.size(); ++gi) {
      const int ns = (int)ctx->plan.groups[gi].mutants.size();
      const ChunkGeom cg = group_geometry(ctx, gi, ns, std::min(ws_bytes, ctx->max_ws_mb << 20));
      if (cg.need_bytes > ws_bytes)
        return ctx->fail(MURE_E_NOMEM, "cluster " + std::to_string(gi) + " needs " + std::to_string(cg.need_bytes) +
                                           " bytes of workspace per chunk; the scratch array holds " +
                                           std::to_string(ws_bytes));
    }
  } else {
    if (!kw) {
      if ((size_t)(M * nwords * 8) > ctx->d_kill.bytes) HIPTRY(ctx->d_kill.alloc((size_t)std::max<int64_t>(M * nwords * 8, 8)));
      kw = ctx->d_kill.as<uint64_t>();
    }
    if ((size_t)(M * 8) > ctx->d_kills.bytes) HIPTRY(ctx->d_kills.alloc((size_t)std::max<int64_t>(M * 8, 8)));
    if ((size_t)(M * mw * 8) > ctx->d_masks.bytes) HIPTRY(ctx->d_masks.alloc((size_t)std::max<int64_t>(M * mw * 8, 8)));
    d_kills = ctx->d_kills.as<int64_t>();
    d_masks = ctx->d_masks.as<unsigned long long>();
  }
  const int64_t timing = ctx->kernel_timing;
  if (noalloc) ctx->kernel_timing = 0;
  struct Restore {
    mure_ctx* c; int64_t t;
    ~Restore() { c->kernel_timing = t; }
  } restore{ctx, timing};
  ctx->stats.launches = 0;
  ctx->stats.group_planes = 0;
  ctx->stats.ms_mmi = 0;
  ctx->stats.gemm_launches = 0;
  ctx->stats.ms_gemm = 0;
  ctx->stats.gemm_macs_algorithmic = 0;
  ctx->stats.gemm_macs_executed = 0;
  for (int f = 0; f < N_FAMILIES; ++f) {
    ctx->stats.kernel_launches[f] = 0;
    ctx->stats.kernel_ms[f] = 0;
    ctx->stats.kernel_macs_algorithmic[f] = 0;
    ctx->stats.kernel_bytes_algorithmic[f] = 0;
  }
  ctx->tevents_used = 0;
  ctx->tevent_family.clear();
  ctx->tevent_mmi.clear();
  HIPTRY(hipEventRecord(ctx->ev0, ctx->stream));
  if (noalloc) {
    // zero fills as kernels (no memset nodes in work a caller may capture)
    HIPTRY(launch_zero_u64(reinterpret_cast<uint64_t*>(ctx->d_nonfinite.p), 1, ctx->stream));
    if (M > 0) HIPTRY(launch_zero_u64(kw, M * nwords, ctx->stream));
  } else {
    HIPTRY(hipMemsetAsync(ctx->d_nonfinite.p, 0, 8, ctx->stream));
    if (M > 0) HIPTRY(hipMemsetAsync(kw, 0, (size_t)(M * nwords * 8), ctx->stream));
  }
  for (int gi = 0; gi < (int)ctx->plan.groups.size(); ++gi) {
    mure_status st = run_group(ctx, gi, 0, (int)ctx->plan.groups[gi].mutants.size(), kw, nullptr, ws, ws_bytes);
    if (st != MURE_OK) return st;
  }
  ScoreArgs sa;
  sa.kill_words = kw;
  sa.nwords = nwords;
  sa.N = N;
  sa.label = ctx->d_label.as<int32_t>();
  sa.mask_words = mw;
  sa.kills = d_kills;
  sa.masks = d_masks;
  HIPTRY(launch_score(sa, (int)M, ctx->stream));
  HIPTRY(hipEventRecord(ctx->ev1, ctx->stream));
  HIPTRY(hipEventSynchronize(ctx->ev1));
  float ms = 0.f;
  HIPTRY(hipEventElapsedTime(&ms, ctx->ev0, ctx->ev1));
  for (size_t i = 0; i + 1 < ctx->tevents_used; i += 2) {
    float t = 0.f;
    HIPTRY(hipEventElapsedTime(&t, ctx->tevents[i], ctx->tevents[i + 1]));
    ctx->stats.ms_gemm += t;
    ctx->stats.kernel_ms[ctx->tevent_family[i / 2]] += t;
    if (ctx->tevent_mmi[i / 2]) ctx->stats.ms_mmi += t;
  }
  ctx->tevents_used = 0;
  ctx->tevent_family.clear();
  ctx->tevent_mmi.clear();
  std::vector<int64_t> kills(M);
  std::vector<unsigned long long> masks(M * mw);
  unsigned long long nonfinite = 0;
  if (M > 0) {
    HIPTRY(hipMemcpy(kills.data(), d_kills, (size_t)(M * 8), hipMemcpyDeviceToHost));
    HIPTRY(hipMemcpy(masks.data(), d_masks, (size_t)(M * mw * 8), hipMemcpyDeviceToHost));
  }
  HIPTRY(hipMemcpy(&nonfinite, ctx->d_nonfinite.p, 8, hipMemcpyDeviceToHost));
  int64_t num = 0, killed = 0;
  for (int64_t m = 0; m < M; ++m) {
    for (int w = 0; w < mw; ++w) num += __builtin_popcountll(masks[m * mw + w]);
    killed += kills[m] > 0;
  }
  if (kills_host && M > 0) std::memcpy(kills_host, kills.data(), (size_t)(M * 8));
  if (score) {
    score->ms_num = num;
    score->ms_den = M * ctx->n_labels;
    score->ms = score->ms_den ? (double)num / (double)score->ms_den : 0.0;
    score->killed_mutants = killed;
    score->n_mutants = M;
    score->n_labels = ctx->n_labels;
    score->n_inputs = N;
    score->nonfinite_logits = (int64_t)nonfinite;
  }
  ctx->stats.ms_run_mutants = ms;
  ctx->stats.macs_vanilla = ctx->plan.macs_vanilla * N;
  ctx->stats.macs_memoized = ctx->plan.macs_memoized * N;
  ctx->stats.macs_algorithmic = ctx->plan.macs_algorithmic * N;
  ctx->stats.macs_executed = ctx->plan.macs_executed * N;
  return MURE_OK;
}

extern "C" {


static mure_status get_logits_impl(mure_ctx* ctx, int32_t mutant_id, float* out_dev) {
  if (!ctx) return MURE_E_INVALID;
  if (ctx->plan_only) return ctx->fail(MURE_E_UNSUPPORTED, "planning-only context");
  if (ctx->state != 3) return ctx->fail(MURE_E_STATE, "run_original must run first");
  if (!out_dev) return ctx->fail(MURE_E_INVALID, "out_dev is NULL");
  if (mutant_id < -1 || mutant_id >= ctx->plan.n_mutants) return ctx->fail(MURE_E_INVALID, "mutant id out of range");
  HIPTRY(hipSetDevice(ctx->device));
  const int64_t bytes = ctx->N * ctx->g.classes() * 4;
  if (mutant_id == -1 || ctx->plan.mutants[mutant_id].mmi < 0) {
    HIPTRY(hipMemcpyAsync(out_dev, ctx->d_logits.p, (size_t)bytes, hipMemcpyDeviceToDevice, ctx->stream));
  } else {
    const MutantPlan& mp = ctx->plan.mutants[mutant_id];
    mure_status st = run_group(ctx, mp.group, mp.slot, mp.slot + 1, nullptr, out_dev);
    if (st != MURE_OK) return st;
  }
  HIPTRY(hipStreamSynchronize(ctx->stream));
  return MURE_OK;
}

static mure_status mutant_plan_impl(const mure_ctx* ctx, int32_t mutant_id, int32_t* mmi, int32_t* group,
                             int32_t* k_nodes, int32_t max_k, int32_t* n_k) {
  if (!ctx) return MURE_E_INVALID;
  if (ctx->state < 2) return const_cast<mure_ctx*>(ctx)->fail(MURE_E_STATE, "apply_mutants first");
  if (mutant_id < 0 || mutant_id >= ctx->plan.n_mutants)
    return const_cast<mure_ctx*>(ctx)->fail(MURE_E_INVALID, "mutant id out of range");
  const MutantPlan& mp = ctx->plan.mutants[mutant_id];
  if (mmi) *mmi = mp.mmi;
  if (group) *group = mp.group;
  if (n_k) *n_k = (int32_t)mp.K.size();
  if (k_nodes)
    for (int i = 0; i < (int)mp.K.size() && i < max_k; ++i) k_nodes[i] = mp.K[i];
  return MURE_OK;
}

static mure_status get_stats_impl(const mure_ctx* ctx, mure_stats* out) {
  if (!ctx || !out) return MURE_E_INVALID;
  *out = ctx->stats;
  out->n_classes = ctx->have_graph ? ctx->g.classes() : 0;
  out->n_inputs = ctx->state == 3 ? ctx->N : 0;
  out->n_mutants = ctx->state >= 2 ? ctx->plan.n_mutants : 0;
  out->n_groups = (int64_t)ctx->plan.groups.size();
  out->n_identity_mutants = ctx->plan.n_identity;
  if (ctx->N == 0) {   // before run_original: per-input ledger
    out->macs_vanilla = ctx->plan.macs_vanilla;
    out->macs_memoized = ctx->plan.macs_memoized;
    out->macs_algorithmic = ctx->plan.macs_algorithmic;
    out->macs_executed = ctx->plan.macs_executed;
  }
  return MURE_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Exported entry points: no C++ exception crosses the interface.  Host
// allocation failures become MURE_E_NOMEM, anything else MURE_E_INVALID, with
// the message in mure_last_error (the call may then have done part of its
// work, as after a device error).
namespace {
mure_status guard_fail(const mure_ctx* ctx, mure_status st, const char* what) noexcept {
  try {
    if (ctx) const_cast<mure_ctx*>(ctx)->err = what;
    else g_create_error = what;
  } catch (...) {
  }
  return st;
}

template <typename F>
mure_status guarded(const mure_ctx* ctx, F&& f) noexcept {
  try {
    return f();
  } catch (const std::bad_alloc&) {
    return guard_fail(ctx, MURE_E_NOMEM, "host memory exhausted");
  } catch (const std::exception& e) {
    return guard_fail(ctx, MURE_E_INVALID, e.what());
  } catch (...) {
    return guard_fail(ctx, MURE_E_INVALID, "unexpected internal error");
  }
}
}  // namespace

extern "C" {

mure_status mure_create(mure_ctx** out, int32_t device, void* hip_stream) {
  return guarded(nullptr, [&] { return create_impl(out, device, hip_stream); });
}

void mure_destroy(mure_ctx* ctx) {
  try {
    destroy_impl(ctx);
  } catch (...) {
  }
}

mure_status mure_set_option(mure_ctx* ctx, const char* name, int64_t value) {
  return guarded(ctx, [&] { return set_option_impl(ctx, name, value); });
}

mure_status mure_load_model(mure_ctx* ctx, const mure_layer* layers, int32_t n_layers, const int32_t in_hwc[3],
                            int32_t dtype, const void* const* weights, const float* const* biases) {
  return guarded(ctx, [&] { return load_model_impl(ctx, layers, n_layers, in_hwc, dtype, weights, biases); });
}

mure_status mure_apply_mutants(mure_ctx* ctx, int32_t n_mutants, const mure_record* records, int64_t n_records) {
  return guarded(ctx, [&] { return apply_mutants_impl(ctx, n_mutants, records, n_records); });
}

mure_status mure_run_original(mure_ctx* ctx, const void* inputs_dev, int64_t n_inputs, const int32_t* labels) {
  return guarded(ctx, [&] { return run_original_impl(ctx, inputs_dev, n_inputs, labels); });
}

mure_status mure_run_mutants(mure_ctx* ctx, uint64_t* kill_bits_dev, int64_t* kills_host, mure_score* score) {
  return guarded(ctx, [&] { return run_mutants_impl(ctx, kill_bits_dev, kills_host, score, false); });
}

mure_status mure_run_mutants_noalloc(mure_ctx* ctx, uint64_t* kill_bits_dev, int64_t* kills_host,
                                     mure_score* score) {
  return guarded(ctx, [&] { return run_mutants_impl(ctx, kill_bits_dev, kills_host, score, true); });
}

mure_status mure_get_logits(mure_ctx* ctx, int32_t mutant_id, float* out_dev) {
  return guarded(ctx, [&] { return get_logits_impl(ctx, mutant_id, out_dev); });
}

mure_status mure_mutant_plan(const mure_ctx* ctx, int32_t mutant_id, int32_t* mmi, int32_t* group,
                             int32_t* k_nodes, int32_t max_k, int32_t* n_k) {
  return guarded(ctx, [&] { return mutant_plan_impl(ctx, mutant_id, mmi, group, k_nodes, max_k, n_k); });
}

mure_status mure_get_stats(const mure_ctx* ctx, mure_stats* out) {
  return guarded(ctx, [&] { return get_stats_impl(ctx, out); });
}

}  // extern "C"
