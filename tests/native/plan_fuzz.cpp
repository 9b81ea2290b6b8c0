// Host-only fuzz driver of the planner (paper_2607_18582_amd/csrc/plan.cpp),
// built with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_plan_sanitized.py.  Seeded random graphs (sequential
// convolutions and dense layers, residual blocks with identity shortcuts,
// depthwise layers, GAP, FLATTEN, token embeddings and LSTMs) and
// random mutation records, valid and invalid, go through build_graph and
// build_plan; on every accepted plan the driver checks what Algorithm 1
// fixes: mmi is the smallest mutated layer, K is exactly the nodes before mmi
// read by a node at or after mmi, and each cluster has one mmi.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <set>
#include <string>
#include <vector>

#include "../../paper_2607_18582_amd/csrc/plan.hpp"

using namespace mure;

namespace {
struct Rng {  // splitmix64
  uint64_t s;
  uint64_t next() {
    uint64_t z = (s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  int below(int n) { return n <= 0 ? 0 : (int)(next() % (uint64_t)n); }
};

Node node(int kind, int src) {
  Node n;
  n.kind = kind;
  n.n_in = kind == K_INPUT ? 0 : 1;
  n.in[0] = src;
  n.in[1] = 0;
  return n;
}

// A random image classifier: returns the node list (input shape in hwc).
std::vector<Node> image_graph(Rng& r, int hwc[3], int& dtype) {
  dtype = r.below(2);
  hwc[0] = hwc[1] = 4 + 4 * r.below(4);
  hwc[2] = 1 + r.below(8);
  std::vector<Node> g{node(K_INPUT, 0)};
  int cur = 0, C = hwc[2], H = hwc[0];
  const int depth = 1 + r.below(5);
  for (int d = 0; d < depth; ++d) {
    const int what = r.below(4);
    if (what == 0 || what == 3) {             // convolution, maybe pooled
      Node n = node(K_CONV, cur);
      n.c_in = C; n.c_out = 4 * (1 + r.below(8)); n.kh = n.kw = 1 + 2 * r.below(2);
      n.pad = n.kh / 2; n.relu = r.below(3);
      if (H >= 4 && r.below(2)) { n.maxpool = 2; H /= 2; }
      g.push_back(n); cur = (int)g.size() - 1; C = n.c_out;
    } else if (what == 1) {                   // residual block, identity shortcut
      Node a = node(K_CONV, cur);
      a.c_in = C; a.c_out = C; a.kh = a.kw = 3; a.pad = 1; a.relu = 1;
      g.push_back(a);
      Node b = node(K_CONV, (int)g.size() - 1);
      b.c_in = C; b.c_out = C; b.kh = b.kw = 3; b.pad = 1;
      g.push_back(b);
      Node add = node(K_ADD, (int)g.size() - 1);
      add.n_in = 2; add.in[1] = cur; add.c_in = C; add.c_out = C; add.relu = 1;
      g.push_back(add); cur = (int)g.size() - 1;
    } else {                                  // depthwise layer
      Node n = node(K_DWCONV, cur);
      n.c_in = C; n.c_out = C; n.kh = n.kw = 3; n.pad = 1; n.relu = 2;
      g.push_back(n); cur = (int)g.size() - 1;
    }
  }
  if (r.below(2)) {
    Node n = node(K_GAP, cur); n.c_in = C; n.c_out = C;
    g.push_back(n); cur = (int)g.size() - 1;
  } else if (r.below(2)) {
    Node n = node(K_FLATTEN, cur); n.c_in = C;
    g.push_back(n); cur = (int)g.size() - 1;
  }
  Node out = node(K_DENSE, cur);
  out.c_out = 2 + r.below(20);
  g.push_back(out);
  return g;
}

std::vector<Node> rnn_graph(Rng& r, int hwc[3], int& dtype) {
  dtype = DT_F32;
  hwc[0] = 1; hwc[1] = 1 + r.below(12); hwc[2] = 1;
  std::vector<Node> g{node(K_INPUT, 0)};
  Node e = node(K_EMBED, 0); e.c_in = 5 + r.below(50); e.c_out = 16 * (1 + r.below(4));
  g.push_back(e);
  Node l1 = node(K_LSTM, 1); l1.c_in = e.c_out; l1.c_out = 16 * (1 + r.below(4)); l1.seq = 1;
  g.push_back(l1);
  Node l2 = node(K_LSTM, 2); l2.c_in = l1.c_out; l2.c_out = 16 * (1 + r.below(4)); l2.seq = 0;
  g.push_back(l2);
  Node out = node(K_DENSE, 3); out.c_out = 2 + r.below(8);
  g.push_back(out);
  return g;
}

// fill the derived input sizes the descriptors need (DENSE c_in = H*W*C of its input)
void fill_dense_inputs(std::vector<Node>& g, int hwc[3]) {
  std::vector<int64_t> elems(g.size(), 0);
  std::vector<int> ch(g.size(), 0);
  int H = hwc[0], W = hwc[1];
  std::vector<int> hh(g.size(), H), ww(g.size(), W);
  ch[0] = hwc[2];
  for (size_t i = 1; i < g.size(); ++i) {
    Node& n = g[i];
    const int s = n.in[0];
    int h = hh[s], w = ww[s], c = ch[s];
    switch (n.kind) {
      case K_CONV: h = (h + 2 * n.pad - n.kh) / n.stride + 1; w = (w + 2 * n.pad - n.kw) / n.stride + 1;
        if (n.maxpool) { h /= 2; w /= 2; } c = n.c_out; break;
      case K_DWCONV: c = n.c_out; break;
      case K_DENSE: n.c_in = h * w * c; h = w = 1; c = n.c_out; break;
      case K_GAP: h = w = 1; break;
      case K_FLATTEN: c = h * w * c; h = w = 1; break;
      case K_EMBED: c = n.c_out; break;
      case K_LSTM: if (!n.seq) w = 1; c = n.c_out; break;
      default: break;
    }
    hh[i] = h; ww[i] = w; ch[i] = c;
  }
}

int fails = 0;
void check(bool ok, const char* what, uint64_t seed) {
  if (!ok) {
    std::printf("FAIL seed %llu: %s\n", (unsigned long long)seed, what);
    ++fails;
  }
}
}  // namespace

int main(int argc, char** argv) {
  const int iters = argc > 1 ? std::atoi(argv[1]) : 3000;
  int accepted = 0, rejected_graphs = 0, rejected_plans = 0;
  for (int it = 0; it < iters; ++it) {
    Rng r{0x1234567ull + (uint64_t)it * 7919ull};
    int hwc[3], dtype = 0;
    std::vector<Node> nodes = r.below(5) == 0 ? rnn_graph(r, hwc, dtype) : image_graph(r, hwc, dtype);
    fill_dense_inputs(nodes, hwc);
    if (r.below(20) == 0) nodes[1 + r.below((int)nodes.size() - 1)].in[0] = (int)nodes.size();   // invalid edge
    Graph g;
    g.nodes = nodes;
    if (!build_graph(g, hwc[0], hwc[1], hwc[2], dtype).empty()) { ++rejected_graphs; continue; }
    std::vector<int> weighted;
    for (int v = 0; v < (int)g.nodes.size(); ++v)
      if (g.nodes[v].weighted()) weighted.push_back(v);
    const int M = r.below(12);
    std::vector<Record> recs;
    int64_t pool = 0;
    for (int m = 0; m < M; ++m) {
      const int k = r.below(4);
      const int op = r.below(5);
      for (int j = 0; j < k; ++j) {
        Record x{};
        x.mutant = r.below(40) == 0 ? M + 1 : m;                         // sometimes out of range
        x.op = r.below(50) == 0 ? 9 : op;
        x.layer = weighted[r.below((int)weighted.size())];
        if (r.below(40) == 0) x.layer = 0;                                // not a weighted node
        const Node& n = g.nodes[x.layer];
        x.neuron = r.below(n.c_out + (r.below(30) == 0 ? 3 : 0));
        x.partner = x.op == OP_NS ? r.below(n.c_out) : -1;
        x.noise_len = (x.op == OP_GF || x.op == OP_WS) ? n.fan_in + (r.below(30) == 0 ? 1 : 0) : 0;
        x.noise_off = pool;
        x.scratch_off = pool + x.noise_len;
        pool += 2 * x.noise_len;
        recs.push_back(x);
      }
    }
    for (int vanilla = 0; vanilla < 2; ++vanilla) {
      Plan plan;
      if (!build_plan(g, M, recs, plan, vanilla != 0).empty()) { ++rejected_plans; continue; }
      ++accepted;
      const uint64_t seed = (uint64_t)it;
      check((int)plan.mutants.size() == M, "one plan per mutant", seed);
      std::set<int> group_mmi;
      for (int m = 0; m < M; ++m) {
        const MutantPlan& mp = plan.mutants[m];
        int lo = 1 << 30;
        for (const Record& x : recs)
          if (x.mutant == m && x.layer < lo) lo = x.layer;
        if (lo == (1 << 30)) { check(mp.mmi == -1, "identity mutant has no mmi", seed); continue; }
        if (vanilla) continue;
        check(mp.mmi == lo, "mmi = smallest mutated layer", seed);
        check(mp.K == boundary(g, mp.mmi), "K of the mutant is the boundary of its mmi", seed);
        std::set<int> want;
        for (int j = mp.mmi; j < (int)g.nodes.size(); ++j)
          for (int q = 0; q < g.nodes[j].n_in; ++q)
            if (g.nodes[j].in[q] < mp.mmi) want.insert(g.nodes[j].in[q]);
        check(std::vector<int>(want.begin(), want.end()) == mp.K, "K = {p < mmi read at or after mmi}", seed);
      }
      for (const Group& gr : plan.groups) {
        check(group_mmi.insert(gr.mmi).second, "one cluster per mmi", seed);
        for (int m : gr.mutants) check(plan.mutants[m].mmi == gr.mmi, "cluster members share mmi", seed);
      }
    }
  }
  std::printf("plans accepted %d, graphs rejected %d, record sets rejected %d, failures %d\n", accepted,
              rejected_graphs, rejected_plans, fails);
  return fails ? 1 : 0;
}
