// Host planner: graph validation, boundaries, clusters, channel patches, ledger.
#include "plan.hpp"

#include <algorithm>
#include <map>
#include <set>
#include <sstream>

namespace mure {

namespace {
std::string fmt_node(int i, const char* what) {
  std::ostringstream s;
  s << "node " << i << ": " << what;
  return s.str();
}
}  // namespace

int64_t Graph::full_macs() const {
  int64_t s = 0;
  for (const Node& n : nodes) s += n.macs;
  return s;
}

int64_t Graph::act_bytes(int v) const {
  const Node& n = nodes[v];
  int64_t es = (v == out() || dtype == DT_F32) ? 4 : 2;
  return n.out_elems() * es;
}

std::string build_graph(Graph& g, int in_h, int in_w, int in_c, int dtype) {
  if (dtype != DT_F32 && dtype != DT_BF16) return "dtype must be MURE_F32 or MURE_BF16";
  if (in_h < 1 || in_w < 1 || in_c < 1) return "in_hwc must be positive";
  const int n = (int)g.nodes.size();
  if (n < 2) return "a model needs an input node and at least one layer";
  g.dtype = dtype;
  for (int i = 0; i < n; ++i) {
    Node& v = g.nodes[i];
    if ((i == 0) != (v.kind == K_INPUT)) return fmt_node(i, "the input must be node 0 and only node 0");
    if (v.kind < K_INPUT || v.kind > K_LSTM) return fmt_node(i, "unknown kind");
    if (i == 0) {
      if (v.n_in != 0) return fmt_node(0, "the input node reads nothing");
      v.H = in_h; v.W = in_w; v.C = in_c;
      if (v.c_out != 0 && v.c_out != in_c) return fmt_node(0, "c_out must equal the input channels");
      continue;
    }
    const int want_in = v.kind == K_ADD ? 2 : 1;
    if (v.n_in != want_in) return fmt_node(i, v.kind == K_ADD ? "ADD reads two nodes" : "reads exactly one node");
    for (int k = 0; k < want_in; ++k)
      if (v.in[k] < 0 || v.in[k] >= i) return fmt_node(i, "inputs must be earlier nodes (topological order)");
    const Node& a = g.nodes[v.in[0]];
    v.inH = a.H; v.inW = a.W; v.inC = a.C;
    if (v.kind != K_CONV && v.maxpool) return fmt_node(i, "only CONV2D may pool");
    if (v.kind != K_ADD && v.shortcut) return fmt_node(i, "only ADD has a shortcut mode");
    if (v.kind != K_LSTM && v.seq) return fmt_node(i, "only LSTM has the seq flag");
    if (v.relu < 0 || v.relu > 2) return fmt_node(i, "relu must be 0 (none), 1 (ReLU) or 2 (ReLU6)");
    switch (v.kind) {
      case K_CONV: {
        if (v.c_in != a.C) return fmt_node(i, "c_in must equal the input channels");
        if (v.c_out < 1 || v.kh < 1 || v.kw < 1 || v.stride < 1 || v.pad < 0)
          return fmt_node(i, "bad convolution geometry");
        if (v.maxpool != 0 && v.maxpool != 2) return fmt_node(i, "maxpool must be 0 or 2");
        v.Hc = (a.H + 2 * v.pad - v.kh) / v.stride + 1;
        v.Wc = (a.W + 2 * v.pad - v.kw) / v.stride + 1;
        if (a.H + 2 * v.pad < v.kh || a.W + 2 * v.pad < v.kw || v.Hc < 1 || v.Wc < 1)
          return fmt_node(i, "kernel larger than the padded input");
        v.H = v.maxpool ? v.Hc / 2 : v.Hc;
        v.W = v.maxpool ? v.Wc / 2 : v.Wc;
        if (v.H < 1 || v.W < 1) return fmt_node(i, "pooling leaves nothing");
        v.C = v.c_out;
        v.fan_in = (int64_t)v.c_in * v.kh * v.kw;
        v.macs = (int64_t)v.Hc * v.Wc * v.c_out * v.fan_in;
        break;
      }
      case K_DWCONV: {
        if (v.c_in != a.C || v.c_out != a.C) return fmt_node(i, "DWCONV keeps the channels (c_in = c_out = C)");
        if (v.kh < 1 || v.kw < 1 || v.stride < 1 || v.pad < 0) return fmt_node(i, "bad convolution geometry");
        v.Hc = (a.H + 2 * v.pad - v.kh) / v.stride + 1;
        v.Wc = (a.W + 2 * v.pad - v.kw) / v.stride + 1;
        if (a.H + 2 * v.pad < v.kh || a.W + 2 * v.pad < v.kw || v.Hc < 1 || v.Wc < 1)
          return fmt_node(i, "kernel larger than the padded input");
        v.H = v.Hc; v.W = v.Wc; v.C = v.c_out;
        v.fan_in = (int64_t)v.kh * v.kw;
        v.macs = (int64_t)v.Hc * v.Wc * v.c_out * v.fan_in;
        break;
      }
      case K_EMBED: {
        if (a.H != 1 || a.C != 1) return fmt_node(i, "EMBED reads a 1 x T x 1 token sequence");
        if (v.c_in < 1 || v.c_out < 1) return fmt_node(i, "EMBED needs a vocabulary (c_in) and a width (c_out)");
        if (v.relu) return fmt_node(i, "EMBED has no activation");
        v.kh = v.kw = v.stride = 1; v.pad = 0;
        v.H = 1; v.W = a.W; v.C = v.c_out;
        v.Hc = v.H; v.Wc = v.W;
        v.fan_in = v.c_in;
        v.macs = 0;
        break;
      }
      case K_LSTM: {
        if (dtype != DT_F32) return fmt_node(i, "LSTM layers need a float32 model");
        if (a.H != 1 || v.c_in != a.C) return fmt_node(i, "LSTM reads a 1 x T x c_in sequence");
        if (v.c_out < 16 || v.c_out > 64 || v.c_out % 16) return fmt_node(i, "LSTM units must be 16, 32, 48 or 64");
        if (v.seq != 0 && v.seq != 1) return fmt_node(i, "seq must be 0 or 1");
        if (v.relu) return fmt_node(i, "LSTM has its own gate activations (relu must be 0)");
        if (lstm_uses_wide(v.c_in, v.c_out) && !lstm_wide_fits(v.c_in, v.c_out))
          return fmt_node(i, "LSTM too wide: c_in + c_out + 1 must be at most 208, and c_in a multiple of 4 "
                             "when the layer's weights exceed 64 KB");
        v.kh = v.kw = v.stride = 1; v.pad = 0;
        v.H = 1; v.W = v.seq ? a.W : 1; v.C = v.c_out;
        v.Hc = v.H; v.Wc = v.W;
        v.fan_in = 4LL * (v.c_in + v.c_out + 1);
        v.macs = (int64_t)a.W * 4 * v.c_out * (v.c_in + v.c_out + 1);
        break;
      }
      case K_DENSE: {
        const int64_t flat = (int64_t)a.H * a.W * a.C;
        if (v.c_in != flat) return fmt_node(i, "c_in must equal H*W*C of the input");
        if (v.c_out < 1) return fmt_node(i, "c_out must be positive");
        if ((v.kh != 0 && v.kh != 1) || (v.kw != 0 && v.kw != 1) || (v.stride != 0 && v.stride != 1) || v.pad != 0)
          return fmt_node(i, "DENSE takes kh=kw=stride=1, pad=0");
        v.kh = v.kw = v.stride = 1;
        v.H = v.W = 1; v.C = v.c_out;
        v.Hc = v.Wc = 1;
        v.fan_in = v.c_in;
        v.macs = (int64_t)v.c_in * v.c_out;
        break;
      }
      case K_ADD: {
        const Node& s = g.nodes[v.in[1]];
        if (v.c_out != a.C) return fmt_node(i, "c_out must equal the channels of in[0]");
        if (v.c_in != s.C) return fmt_node(i, "c_in must equal the channels of in[1]");
        if (v.shortcut == 0) {
          if (s.H != a.H || s.W != a.W || s.C != a.C) return fmt_node(i, "identity shortcut needs equal shapes");
        } else if (v.shortcut == 1) {
          if ((s.H + 1) / 2 != a.H || (s.W + 1) / 2 != a.W || s.C > a.C)
            return fmt_node(i, "option-A shortcut: in[1] must be 2x the size with at most C channels");
        } else {
          return fmt_node(i, "shortcut must be 0 or 1");
        }
        if (v.kh > 1 || v.kw > 1 || v.stride > 1 || v.pad) return fmt_node(i, "ADD has no geometry");
        v.H = a.H; v.W = a.W; v.C = a.C;
        break;
      }
      case K_GAP:
        if (v.c_in != a.C || v.c_out != a.C) return fmt_node(i, "GAP keeps the channels (c_in = c_out = C)");
        v.H = v.W = 1; v.C = a.C;
        break;
      case K_FLATTEN:
        v.H = v.W = 1; v.C = a.H * a.W * a.C;
        if (v.c_out != 0 && v.c_out != v.C) return fmt_node(i, "c_out must be H*W*C");
        break;
    }
  }
  if (g.nodes.back().H != 1 || g.nodes.back().W != 1) return "the output node must be 1x1xC";
  if (g.nodes.back().kind == K_FLATTEN) return "the output node must compute its logits (not a FLATTEN view)";
  if (g.nodes.back().C < 2 || g.nodes.back().C > 512) return "the output needs 2 to 512 classes";
  // every node but the output must be read by some later node
  std::vector<int> used(n, 0);
  for (int i = 1; i < n; ++i)
    for (int k = 0; k < g.nodes[i].n_in; ++k) used[g.nodes[i].in[k]] = 1;
  for (int i = 0; i + 1 < n; ++i)
    if (!used[i]) return fmt_node(i, "is not read by any node (the output must be the last node)");
  return "";
}

int node_family(const Graph& g, int v) {
  const Node& n = g.nodes[v];
  if (n.kind == K_DWCONV) return FAM_DW;
  if (n.kind == K_EMBED) return FAM_EMBED;
  if (n.kind == K_LSTM) return FAM_LSTM;
  if (n.kind == K_DENSE) {
    const int vec = g.dtype == DT_F32 ? 4 : 8;       // 16-byte rows
    return (n.c_in % vec == 0 && n.c_out <= 256) ? FAM_DENSE : FAM_GEMM;
  }
  if (n.kind != K_CONV) return -1;
  const int P = n.maxpool ? 4 * n.H * n.W : n.Hc * n.Wc;
  if (n.c_out < 16 && valu_lds_bytes(n.inH, n.inW, n.inC, n.pad, n.H * n.W, n.c_out, n.fan_in) <= 48 * 1024)
    return FAM_VALU;
  if (g.dtype == DT_F32 && n.c_out <= 64 &&
      conv_lds_bytes(n.inH, n.inW, n.inC, n.pad, P, n.c_out, n.fan_in) <= 48 * 1024)
    return FAM_LDS;
  // halo tiles are 32 or 64 columns wide: 16-column outputs stay on the
  // gather kernel, which wastes no MFMA columns on them
  if (g.dtype == DT_BF16 && v != g.out() && n.c_out % 32 == 0 &&
      conv_halo_fits(n.inH, n.inW, n.inC, n.kh, n.kw, n.stride, n.pad))
    return FAM_HALO;
  if (g.dtype == DT_BF16 && n.inC % 8 == 0 && n.kh <= 15 && n.kw <= 15 && n.fan_in <= 8192 &&
      P % 4 == 0 && ((int64_t)n.kh * n.inW + n.kw) * n.inC < (1 << 24))
    return FAM_BIG;
  return FAM_GEMM;
}

// The ADD node that reads convolution v as its first input when nothing else
// reads v (conv_b of a residual block): the pair runs as one launch whose
// epilogue adds the shortcut.  -1 if v is not such a convolution.
int fused_add_of(const Graph& g, int v) {
  const Node& n = g.nodes[v];
  const int fam = node_family(g, v);
  if (n.kind != K_CONV || n.maxpool || (fam != FAM_BIG && fam != FAM_HALO)) return -1;
  int reader = -1, count = 0;
  for (int j = v + 1; j < (int)g.nodes.size(); ++j)
    for (int k = 0; k < g.nodes[j].n_in; ++k)
      if (g.nodes[j].in[k] == v) { reader = j; ++count; }
  if (count != 1 || g.nodes[reader].kind != K_ADD || g.nodes[reader].in[0] != v) return -1;
  if (fam == FAM_HALO && reader == g.out()) return -1;   // the halo kernel stores bf16 only
  return reader;
}

std::vector<int> boundary(const Graph& g, int mmi) {
  std::set<int> K;
  for (int j = mmi; j < (int)g.nodes.size(); ++j)
    for (int k = 0; k < g.nodes[j].n_in; ++k)
      if (g.nodes[j].in[k] < mmi) K.insert(g.nodes[j].in[k]);
  return std::vector<int>(K.begin(), K.end());
}

std::string build_plan(const Graph& g, int n_mutants, const std::vector<Record>& recs, Plan& plan,
                       bool vanilla) {
  std::ostringstream err;
  if (n_mutants < 0) return "n_mutants must be >= 0";
  const int n = (int)g.nodes.size();
  for (size_t r = 0; r < recs.size(); ++r) {
    const Record& x = recs[r];
    if (x.mutant < 0 || x.mutant >= n_mutants) { err << "record " << r << ": mutant out of range"; return err.str(); }
    if (x.layer < 0 || x.layer >= n || !g.nodes[x.layer].weighted()) {
      err << "record " << r << ": layer " << x.layer << " is not a DENSE/CONV2D node"; return err.str();
    }
    const Node& v = g.nodes[x.layer];
    if (x.neuron < 0 || x.neuron >= v.c_out) { err << "record " << r << ": neuron out of range"; return err.str(); }
    if (x.op < OP_GF || x.op > OP_WS) { err << "record " << r << ": unknown operator " << x.op; return err.str(); }
    if (x.op == OP_NS && (x.partner < 0 || x.partner >= v.c_out || x.partner == x.neuron)) {
      err << "record " << r << ": neuron switch needs a partner in [0, c_out) other than the neuron"; return err.str();
    }
    if ((x.op == OP_GF || x.op == OP_WS) && x.noise_len != v.fan_in) {
      err << "record " << r << ": parameter length " << x.noise_len << " != fan-in " << v.fan_in; return err.str();
    }
  }
  Plan p;
  p.n_mutants = n_mutants;
  p.mutants.assign(n_mutants, MutantPlan());
  std::vector<std::vector<int>> by_mutant(n_mutants);
  for (size_t r = 0; r < recs.size(); ++r) by_mutant[recs[r].mutant].push_back((int)r);

  std::map<int, std::vector<int>> groups;   // mmi -> mutants
  for (int m = 0; m < n_mutants; ++m) {
    MutantPlan& mp = p.mutants[m];
    const std::vector<int>& rs = by_mutant[m];
    if (rs.empty()) { p.n_identity++; continue; }
    std::set<int> mu;
    for (int r : rs) mu.insert(recs[r].layer);
    mp.layers.assign(mu.begin(), mu.end());
    mp.mmi = mp.layers.front();
    if (vanilla) {                       // start at the first weighted node
      int first = 1;
      while (!g.nodes[first].weighted()) ++first;
      mp.mmi = first;
    }
    mp.K = boundary(g, mp.mmi);
    std::set<int> fuzzed;
    // a switch on a depthwise layer pairs each filter with the other
    // channel's input, so it is recomputed like a fuzz (its output is not a
    // channel exchange of the original's)
    const bool dw = g.nodes[mp.mmi].kind == K_DWCONV;
    for (int r : rs)
      if (recs[r].layer == mp.mmi && (recs[r].op == OP_GF || recs[r].op == OP_NAI || recs[r].op == OP_WS ||
                                      (dw && recs[r].op == OP_NS))) {
        mp.recompute = true;
        fuzzed.insert(recs[r].neuron);
        if (recs[r].op == OP_NS) fuzzed.insert(recs[r].partner);
      }
    // an LSTM unit feeds every unit's next step: any record there changes
    // the whole layer, which is recomputed
    if (g.nodes[mp.mmi].kind == K_LSTM) {
      mp.recompute = true;
      for (int c = 0; c < g.nodes[mp.mmi].c_out; ++c) fuzzed.insert(c);
    }
    if (vanilla) mp.recompute = true;    // the whole first layer, with its own weights
    mp.touched = (int64_t)fuzzed.size();
    const int C = g.nodes[mp.mmi].c_out;
    mp.chmap.resize(C);
    for (int c = 0; c < C; ++c) mp.chmap[c] = c;
    if (!mp.recompute) {
      // effect-block / switch records only: every CONV2D/DENSE epilogue here is
      // per channel (bias, ReLU, pool), so the mutated node's output is the
      // original's with channels zeroed or exchanged.
      for (int r : rs) {
        if (recs[r].layer != mp.mmi) continue;
        if (recs[r].op == OP_NEB) mp.chmap[recs[r].neuron] = -1;
        else std::swap(mp.chmap[recs[r].neuron], mp.chmap[recs[r].partner]);
      }
    } else {
      std::set<int> tl;
      for (int r : rs) {
        if (recs[r].layer != mp.mmi) continue;
        tl.insert(recs[r].neuron);
        if (recs[r].op == OP_NS) tl.insert(recs[r].partner);
      }
      mp.touched_list.assign(tl.begin(), tl.end());
    }
    if (vanilla) {                       // layers before the first mutated one keep the original
      mp.chmap.assign(g.nodes[mp.mmi].c_out, 0);
      for (int c = 0; c < (int)mp.chmap.size(); ++c) mp.chmap[c] = c;
      mp.touched_list.clear();
    }
    for (int l : mp.layers) {
      CowCopy cc;
      cc.mutant = m; cc.layer = l;
      for (int r : rs) if (recs[r].layer == l) cc.records.push_back(r);
      p.cows.push_back(cc);
    }
    groups[mp.mmi].push_back(m);
  }
  std::set<int> cache;
  std::vector<int64_t> prefix(n + 1, 0);
  for (int v = 0; v < n; ++v) prefix[v + 1] = prefix[v] + g.nodes[v].macs;
  const int64_t full = prefix[n];
  for (auto& kv : groups) {
    Group gr;
    gr.mmi = kv.first;
    gr.K = boundary(g, gr.mmi);
    for (int m : kv.second) if (p.mutants[m].recompute) gr.mutants.push_back(m);
    gr.n_recompute = (int)gr.mutants.size();
    for (int m : kv.second) if (!p.mutants[m].recompute) gr.mutants.push_back(m);
    // delta at mmi: only the channels the fuzz / inverse / shuffle records
    // changed are recomputed (per slot on the VALU and depthwise kernels, or
    // one gathered-column GEMM over the shared cached input for the MFMA
    // families); the sequence layers recompute whole nodes
    {
      const int fam = node_family(g, gr.mmi);
      gr.delta = !vanilla && gr.n_recompute > 0 &&
                 (fam == FAM_VALU || fam == FAM_LDS || fam == FAM_DENSE || fam == FAM_BIG || fam == FAM_DW ||
                  fam == FAM_GEMM || fam == FAM_HALO);
    }
    // virtual mmi output: every consumer is an LDS convolution or a dense layer
    gr.virt = gr.mmi != g.out();
    for (int v = gr.mmi + 1; v < n && gr.virt; ++v)
      for (int k = 0; k < g.nodes[v].n_in; ++k)
        if (g.nodes[v].in[k] == gr.mmi) {
          const int f = node_family(g, v);
          if (!(f == FAM_LDS || (f == FAM_DENSE && g.nodes[v].c_in <= 4096))) gr.virt = false;
        }
    // channel-group reads (halo kernel): every consumer of mmi is a halo
    // convolution reading it as its only input, or an identity-shortcut ADD
    // fused into a halo convolution
    if (!gr.virt && !vanilla && gr.mmi != g.out() && g.dtype == DT_BF16 && g.nodes[gr.mmi].c_out % 8 == 0 &&
        (gr.delta || gr.n_recompute == 0)) {
      bool ok = true, any = false;
      for (int v = gr.mmi + 1; v < n && ok; ++v) {
        const Node& nv = g.nodes[v];
        for (int k = 0; k < nv.n_in; ++k) {
          if (nv.in[k] != gr.mmi) continue;
          if (k == 0 && nv.n_in == 1 && node_family(g, v) == FAM_HALO) {
            any = true;
          } else if (!(nv.kind == K_ADD && k == 1 && nv.shortcut == 0 && node_family(g, nv.in[0]) == FAM_HALO &&
                       fused_add_of(g, nv.in[0]) == v)) {
            ok = false;
          }
        }
      }
      gr.vhalo = ok && any;
    }
    if (gr.virt || gr.vhalo) {
      const int C = g.nodes[gr.mmi].c_out;
      gr.T = 0;
      if (gr.n_recompute > 0) {
        if (gr.delta) {
          for (int s = 0; s < gr.n_recompute; ++s)
            gr.T = std::max(gr.T, (int)p.mutants[gr.mutants[s]].touched_list.size());
        } else {
          gr.T = C;
        }
      }
      gr.vchmap.resize(gr.mutants.size() * C);
      for (size_t s = 0; s < gr.mutants.size(); ++s) {
        const MutantPlan& mp = p.mutants[gr.mutants[s]];
        int* row = &gr.vchmap[s * C];
        for (int c = 0; c < C; ++c) row[c] = mp.chmap[c];
        if ((int)s < gr.n_recompute) {
          if (gr.delta)
            for (size_t t = 0; t < mp.touched_list.size(); ++t) row[mp.touched_list[t]] = -2 - (int)t;
          else
            for (int c = 0; c < C; ++c) row[c] = -2 - c;
        }
      }
    }
    for (int k : gr.K) cache.insert(k);
    if (gr.n_recompute < (int)gr.mutants.size() || gr.delta || gr.virt) cache.insert(gr.mmi);
    const int gi = (int)p.groups.size();
    for (size_t s = 0; s < gr.mutants.size(); ++s) {
      p.mutants[gr.mutants[s]].group = gi;
      p.mutants[gr.mutants[s]].slot = (int)s;
    }
    const Node& l = g.nodes[gr.mmi];
    const int64_t after = full - prefix[gr.mmi + 1];
    p.macs_memoized += prefix[gr.mmi] + (int64_t)gr.mutants.size() * (full - prefix[gr.mmi]);
    for (int m : gr.mutants) {
      const MutantPlan& mp = p.mutants[m];
      p.macs_vanilla += full;
      p.macs_algorithmic += mp.touched * (l.macs / l.c_out) + after;
      const int64_t at_mmi = !mp.recompute ? 0
                             : gr.delta ? (int64_t)mp.touched_list.size() * (l.macs / l.c_out) : l.macs;
      p.macs_executed += at_mmi + after;
    }
    p.groups.push_back(std::move(gr));
  }
  p.cache_nodes.assign(cache.begin(), cache.end());
  plan = std::move(p);
  return "";
}

}  // namespace mure
