// ea_logical.cpp -- logical optimization (Section 4): the choice of a
// join-agg spec for every abstract operator of a computation over p
// processors, by dynamic programming over output tilings (Section 4.2,
// Algorithm "Logical optimization"), with the communication proxy of
// Section 4.3 and the tree cuts of Section 4.5.
//
// A spec decomposes each shardable letter into near-equal intervals; the
// counts multiply to p.  Its function specifications are the cells of that
// grid, so the proxy's sums have closed forms: the k-th inputs of all p
// cells hold |X_k| * p / (product of input k's counts) numbers (each block of
// the input's tiling appears once per cell of the other letters), and every
// output block appears p / (product of the output's counts) times.
//
// The repartition sub-cost of input k depends on that input's tiling only,
// so the joint minimum over (T_1, ..., T_n) of B(J) is the sum of per-input
// minima: the table is filled in O(s t n) per operator.
#include <algorithm>
#include <cstring>
#include <vector>

#include "ea_internal.h"

namespace ea {
namespace {

using Tiling = std::vector<int32_t>;  // interval count of every dim of a tensor

struct Op {
  Spec sp;
  int n_letters = 0;
  char letter[kMaxLetters] = {};
  int64_t ext[kMaxLetters] = {};
  bool shard[kMaxLetters] = {};
  int input[EA_LOP_MAX_INPUTS] = {};
  int dim_letter[kMaxOps][kMaxRank] = {};  // operand (inputs, then output), dim -> letter
  int64_t size[kMaxOps] = {};              // elements of every operand
  std::vector<std::vector<int32_t>> specs; // counts per letter
};

struct Entry {           // Opt[op, T] and its choice
  Tiling t;
  int64_t opt = 0;
  int spec = -1;
  std::vector<int> in_choice;  // per input: index into the producer's candidates (-1: none)
};

Tiling tiling_of(const Op& o, int operand, const std::vector<int32_t>& c) {
  Tiling t(o.sp.rank[operand]);
  for (int d = 0; d < o.sp.rank[operand]; ++d) t[d] = c[o.dim_letter[operand][d]];
  return t;
}

// join and aggregation sub-costs of a spec (the repartition one depends on
// the input tilings)
int64_t join_agg_cost(const Op& o, const std::vector<int32_t>& c, int64_t p) {
  int64_t cost = 0;
  for (int k = 0; k <= o.sp.n_in; ++k) {
    int64_t prod = 1;
    for (int d = 0; d < o.sp.rank[k]; ++d) prod *= c[o.dim_letter[k][d]];
    if (k < o.sp.n_in) cost += o.size[k] * (p / prod);
    else cost += (p / prod - 1) * o.size[k];
  }
  return cost;
}

// every assignment of counts to the shardable letters with product p, each
// count at most the letter's extent (letters in order, counts ascending)
int enumerate_specs(Op& o, int64_t p) {
  std::vector<int32_t> c(o.n_letters, 1);
  bool overflow = false;
  auto rec = [&](auto&& self, int l, int64_t rem) -> void {
    if (overflow) return;
    if (l == o.n_letters) {
      if (rem == 1) {
        if (o.specs.size() >= ((size_t)1 << 20)) overflow = true;
        else o.specs.push_back(c);
      }
      return;
    }
    if (!o.shard[l]) {
      c[l] = 1;
      self(self, l + 1, rem);
      return;
    }
    for (int64_t v = 1; v <= rem && v <= o.ext[l]; ++v) {
      if (rem % v) continue;
      c[l] = (int32_t)v;
      self(self, l + 1, rem / v);
    }
    c[l] = 1;
  };
  rec(rec, 0, p);
  if (overflow) return fail(EA_ERR_UNSUPPORTED, "more than 2^20 join-agg specs for one operator");
  return EA_OK;
}

}  // namespace
}  // namespace ea

using namespace ea;

extern "C" int ea_logical_plan(int32_t n_ops, const ea_lop* lops, int64_t p, int32_t* counts, int64_t* cost) {
  if (n_ops < 1 || !lops || !counts || !cost) return fail(EA_ERR_ARG, "ea_logical_plan: bad arguments");
  if (p < 1) return fail(EA_ERR_ARG, "ea_logical_plan: p = %lld", (long long)p);
  std::vector<Op> ops((size_t)n_ops);
  for (int i = 0; i < n_ops; ++i) {
    Op& o = ops[(size_t)i];
    const ea_lop& L = lops[i];
    int e = parse_spec(L.spec, &o.sp);
    if (e) return e;
    if (!L.extents) return fail(EA_ERR_ARG, "operator %d: NULL extents", i);
    for (int k = 0; k <= o.sp.n_in; ++k)
      for (int d = 0; d < o.sp.rank[k]; ++d) {
        const char ch = o.sp.let[k][d];
        int l = 0;
        while (l < o.n_letters && o.letter[l] != ch) ++l;
        if (l == o.n_letters) {
          if (o.n_letters == kMaxLetters) return fail(EA_ERR_SPEC, "operator %d: more than %d letters", i, kMaxLetters);
          o.letter[o.n_letters] = ch;
          o.ext[o.n_letters] = L.extents[o.n_letters];
          if (o.ext[o.n_letters] < 1) return fail(EA_ERR_ARG, "operator %d: extent of '%c' below 1", i, ch);
          o.shard[o.n_letters] = !L.shardable || strchr(L.shardable, ch) != nullptr;
          ++o.n_letters;
        }
        o.dim_letter[k][d] = l;
      }
    if (L.shardable)
      for (const char* q = L.shardable; *q; ++q)
        if (!memchr(o.letter, *q, (size_t)o.n_letters))
          return fail(EA_ERR_SPEC, "operator %d: shardable letter '%c' not in its spec", i, *q);
    for (int k = 0; k <= o.sp.n_in; ++k) {
      o.size[k] = 1;
      for (int d = 0; d < o.sp.rank[k]; ++d) o.size[k] *= o.ext[o.dim_letter[k][d]];
    }
    for (int k = 0; k < o.sp.n_in; ++k) {
      const int pr = L.input[k];
      o.input[k] = pr;
      if (pr < -1 || pr >= i) return fail(EA_ERR_ARG, "operator %d input %d: producer %d", i, k, pr);
      if (pr >= 0) {  // the producer's output is this input: same shape
        const Op& q = ops[(size_t)pr];
        const int qo = q.sp.n_in;
        bool same = q.sp.rank[qo] == o.sp.rank[k];
        for (int d = 0; same && d < o.sp.rank[k]; ++d)
          same = q.ext[q.dim_letter[qo][d]] == o.ext[o.dim_letter[k][d]];
        if (!same) return fail(EA_ERR_SPEC, "operator %d input %d: shape differs from operator %d's output", i, k, pr);
      }
    }
    e = enumerate_specs(o, p);
    if (e) return e;
    if (o.specs.empty())
      return fail(EA_ERR_UNSUPPORTED, "operator %d ('%s'): no decomposition into %lld near-equal pieces", i, L.spec,
                  (long long)p);
  }

  // trees (Section 4.5): an output consumed exactly once is a tree edge
  std::vector<std::vector<std::pair<int, int>>> consumers((size_t)n_ops);  // (consumer, input)
  for (int i = 0; i < n_ops; ++i)
    for (int k = 0; k < ops[(size_t)i].sp.n_in; ++k)
      if (ops[(size_t)i].input[k] >= 0) consumers[(size_t)ops[(size_t)i].input[k]].push_back({i, k});
  auto in_tree_edge = [&](int prod) { return prod >= 0 && consumers[(size_t)prod].size() == 1; };
  std::vector<int> tree_of((size_t)n_ops, -1);
  std::vector<int> roots;
  for (int i = n_ops - 1; i >= 0; --i) {
    if (in_tree_edge(i)) continue;
    roots.push_back(i);
    std::vector<int> stack{i};
    while (!stack.empty()) {
      const int x = stack.back();
      stack.pop_back();
      tree_of[(size_t)x] = i;
      for (int k = 0; k < ops[(size_t)x].sp.n_in; ++k)
        if (in_tree_edge(ops[(size_t)x].input[k])) stack.push_back(ops[(size_t)x].input[k]);
    }
  }
  std::vector<int> tsize((size_t)n_ops, 0);
  for (int i = 0; i < n_ops; ++i) ++tsize[(size_t)tree_of[(size_t)i]];
  std::stable_sort(roots.begin(), roots.end(), [&](int a, int b) {
    return tsize[(size_t)a] != tsize[(size_t)b] ? tsize[(size_t)a] > tsize[(size_t)b] : a < b;
  });

  std::vector<int> chosen((size_t)n_ops, -1);       // spec index of every operator
  std::vector<Tiling> out_tiling((size_t)n_ops);    // its output tiling
  std::vector<bool> fixed((size_t)n_ops, false);
  std::vector<std::vector<Entry>> cand((size_t)n_ops);
  for (int root : roots) {
    // bottom-up over the tree's operators (producers have lower indices)
    for (int i = 0; i < n_ops; ++i) {
      if (tree_of[(size_t)i] != root) continue;
      const Op& o = ops[(size_t)i];
      std::vector<Entry>& cd = cand[(size_t)i];
      cd.clear();
      for (int j = 0; j < (int)o.specs.size(); ++j) {
        const std::vector<int32_t>& c = o.specs[(size_t)j];
        int64_t b = join_agg_cost(o, c, p);
        std::vector<int> choice((size_t)o.sp.n_in, -1);
        for (int k = 0; k < o.sp.n_in; ++k) {
          const int pr = o.input[k];
          if (pr < 0) continue;  // computation input: materialised as J needs
          const Tiling need = tiling_of(o, k, c);
          if (tree_of[(size_t)pr] == root) {  // in the tree: the producer's best candidate
            int best = -1;
            int64_t bv = 0;
            const std::vector<Entry>& pc = cand[(size_t)pr];
            for (int t = 0; t < (int)pc.size(); ++t) {
              const int64_t v = pc[(size_t)t].opt + (pc[(size_t)t].t != need ? o.size[k] : 0);
              if (best < 0 || v < bv) {
                best = t;
                bv = v;
              }
            }
            choice[(size_t)k] = best;
            b += bv;
          } else if (fixed[(size_t)pr]) {  // from a tree already optimised
            b += out_tiling[(size_t)pr] != need ? o.size[k] : 0;
          }  // else from a tree not optimised yet: a computation input for now
        }
        const Tiling t = tiling_of(o, o.sp.n_in, c);
        auto it = std::find_if(cd.begin(), cd.end(), [&](const Entry& en) { return en.t == t; });
        if (it == cd.end()) {
          cd.push_back(Entry{t, b, j, choice});
        } else if (b < it->opt) {
          it->opt = b;
          it->spec = j;
          it->in_choice = choice;
        }
      }
    }
    // the root's tiling: its table entry plus the repartitions of consumers
    // already fixed in other trees
    const Op& ro = ops[(size_t)root];
    int best = -1;
    int64_t bv = 0;
    for (int t = 0; t < (int)cand[(size_t)root].size(); ++t) {
      int64_t v = cand[(size_t)root][(size_t)t].opt;
      for (const auto& ck : consumers[(size_t)root]) {
        if (!fixed[(size_t)ck.first]) continue;
        const Op& co = ops[(size_t)ck.first];
        if (tiling_of(co, ck.second, co.specs[(size_t)chosen[(size_t)ck.first]]) != cand[(size_t)root][(size_t)t].t)
          v += ro.size[ro.sp.n_in];
      }
      if (best < 0 || v < bv) {
        best = t;
        bv = v;
      }
    }
    // assign: walk back from the root through the recorded choices
    std::vector<std::pair<int, int>> stack{{root, best}};
    while (!stack.empty()) {
      const auto [x, t] = stack.back();
      stack.pop_back();
      const Entry& en = cand[(size_t)x][(size_t)t];
      chosen[(size_t)x] = en.spec;
      out_tiling[(size_t)x] = en.t;
      fixed[(size_t)x] = true;
      for (int k = 0; k < ops[(size_t)x].sp.n_in; ++k)
        if (en.in_choice[(size_t)k] >= 0) stack.push_back({ops[(size_t)x].input[k], en.in_choice[(size_t)k]});
    }
  }

  // the plan's total cost under the model, and the counts
  int64_t total = 0;
  for (int i = 0; i < n_ops; ++i) {
    const Op& o = ops[(size_t)i];
    const std::vector<int32_t>& c = o.specs[(size_t)chosen[(size_t)i]];
    total += join_agg_cost(o, c, p);
    for (int k = 0; k < o.sp.n_in; ++k)
      if (o.input[k] >= 0 && out_tiling[(size_t)o.input[k]] != tiling_of(o, k, c)) total += o.size[k];
    for (int l = 0; l < kMaxLetters; ++l) counts[(int64_t)i * kMaxLetters + l] = l < o.n_letters ? c[(size_t)l] : 0;
  }
  *cost = total;
  return ok();
}
