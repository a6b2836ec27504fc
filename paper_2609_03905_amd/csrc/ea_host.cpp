// ea_host.cpp -- libea host side: relation handles, layout, validation, spec
// parsing, join analysis, the plan cache and kernel dispatch.
//
// Nothing here computes a result: every step of a join-agg or repartition runs
// in the HIP kernels.  This file decides, for each call, which kernel runs on
// which blocks and tuples, and builds the device plan those kernels read.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <sstream>
#include <string>
#include <vector>

#include "ea_internal.h"

using namespace ea;

struct ea_relation {
  int32_t rank = 0;
  int32_t dtype = 0;
  int64_t shape[kMaxRank] = {};
  int32_t nb[kMaxRank] = {};
  std::vector<int64_t> splits[kMaxRank];
  std::vector<int64_t> off;  // byte offset of every block
  int64_t nblocks = 0;
  int64_t nbytes = 0;
  void* data = nullptr;
  int64_t capacity = 0;
};

// ---------------------------------------------------------------------------
// errors (shared with the other host sources through ea_internal.h)
// ---------------------------------------------------------------------------
namespace ea {
thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[1024];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return EA_OK;
}
}  // namespace ea

namespace {

#define EA_HIP_TRY(expr)                                                              \
  do {                                                                                \
    hipError_t e_ = (expr);                                                           \
    if (e_ != hipSuccess)                                                             \
      return fail(EA_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));         \
  } while (0)

int dtype_size(int32_t dt) {
  switch (dt) {
    case EA_F32: return 4;
    case EA_BF16: return 2;
    case EA_F16: return 2;
    default: return EA_ERR_DTYPE;
  }
}

int64_t align256(int64_t x) { return (x + 255) / 256 * 256; }

// ---------------------------------------------------------------------------
// partitions and layout
// ---------------------------------------------------------------------------
int check_partition(int32_t rank, const int64_t* shape, const int32_t* nblocks,
                    const int64_t* splits) {
  if (rank < 1 || rank > kMaxRank) return fail(EA_ERR_ARG, "rank %d outside [1, %d]", rank, kMaxRank);
  if (!shape || !nblocks || !splits) return fail(EA_ERR_ARG, "NULL shape, nblocks or splits");
  const int64_t* s = splits;
  int64_t total_blocks = 1;
  for (int d = 0; d < rank; ++d) {
    if (shape[d] < 1 || shape[d] > INT32_MAX)
      return fail(EA_ERR_ARG, "extent %lld of dim %d outside [1, 2^31)", (long long)shape[d], d);
    if (nblocks[d] < 1 || nblocks[d] > shape[d])
      return fail(EA_ERR_PARTITION, "dim %d: %d blocks for extent %lld", d, nblocks[d],
                  (long long)shape[d]);
    if (s[0] != 0) return fail(EA_ERR_PARTITION, "dim %d: first split point is not 0", d);
    for (int b = 0; b < nblocks[d]; ++b)
      if (s[b + 1] <= s[b])
        return fail(EA_ERR_PARTITION, "dim %d: split points not strictly increasing at %d", d, b);
    if (s[nblocks[d]] != shape[d])
      return fail(EA_ERR_PARTITION, "dim %d: last split point %lld is not the extent %lld", d,
                  (long long)s[nblocks[d]], (long long)shape[d]);
    total_blocks *= nblocks[d];
    if (total_blocks > INT32_MAX) return fail(EA_ERR_ARG, "too many blocks");
    s += nblocks[d] + 1;
  }
  return EA_OK;
}

void fill_layout(ea_relation* r) {
  r->nblocks = 1;
  for (int d = 0; d < r->rank; ++d) r->nblocks *= r->nb[d];
  r->off.assign((size_t)r->nblocks, 0);
  const int es = dtype_size(r->dtype);
  int64_t pos = 0, end = 0;
  int32_t c[kMaxRank] = {};
  for (int64_t b = 0; b < r->nblocks; ++b) {
    int64_t n = 1;
    for (int d = 0; d < r->rank; ++d) n *= r->splits[d][c[d] + 1] - r->splits[d][c[d]];
    pos = align256(pos);
    r->off[(size_t)b] = pos;
    end = pos + n * es;
    pos = end;
    for (int d = r->rank - 1; d >= 0; --d) {  // next block coordinates, row-major
      if (++c[d] < r->nb[d]) break;
      c[d] = 0;
    }
  }
  r->nbytes = end;
}

void block_coords(const ea_relation* r, int64_t b, int32_t* c) {
  for (int d = r->rank - 1; d >= 0; --d) {
    c[d] = (int32_t)(b % r->nb[d]);
    b /= r->nb[d];
  }
}

std::vector<DevBlk> dev_blocks(const ea_relation* r) {
  std::vector<DevBlk> v((size_t)r->nblocks);
  int32_t c[kMaxRank];
  for (int64_t b = 0; b < r->nblocks; ++b) {
    block_coords(r, b, c);
    DevBlk& x = v[(size_t)b];
    memset(&x, 0, sizeof(x));
    x.off = r->off[(size_t)b];
    for (int d = 0; d < r->rank; ++d) {
      x.lo[d] = (int32_t)r->splits[d][c[d]];
      x.ext[d] = (int32_t)(r->splits[d][c[d] + 1] - r->splits[d][c[d]]);
    }
  }
  return v;
}

}  // namespace

// ---------------------------------------------------------------------------
// einsum spec
// ---------------------------------------------------------------------------
namespace ea {
bool is_letter(char ch) { return (ch >= 'a' && ch <= 'z') || (ch >= 'A' && ch <= 'Z'); }

int parse_spec(const char* s, Spec* sp) {
  if (!s) return fail(EA_ERR_ARG, "NULL spec");
  *sp = Spec();
  const char* arrow = strstr(s, "->");
  if (!arrow) return fail(EA_ERR_SPEC, "spec '%s' has no '->'", s);
  int op = 0, r = 0;
  auto add = [&](char ch) -> int {
    if (!is_letter(ch)) return fail(EA_ERR_SPEC, "spec '%s': bad character '%c'", s, ch);
    if (r >= kMaxRank) return fail(EA_ERR_SPEC, "spec '%s': operand rank above %d", s, kMaxRank);
    for (int i = 0; i < r; ++i)
      if (sp->let[op][i] == ch) return fail(EA_ERR_SPEC, "spec '%s': letter '%c' repeats in an operand", s, ch);
    sp->let[op][r++] = ch;
    return EA_OK;
  };
  for (const char* p = s; p != arrow; ++p) {
    if (*p == ',') {
      if (r == 0) return fail(EA_ERR_SPEC, "spec '%s': empty operand", s);
      if (op + 1 >= kMaxIn) return fail(EA_ERR_SPEC, "spec '%s': more than %d inputs", s, kMaxIn);
      sp->rank[op++] = r;
      r = 0;
      continue;
    }
    int e = add(*p);
    if (e) return e;
  }
  if (r == 0) return fail(EA_ERR_SPEC, "spec '%s': empty operand", s);
  sp->rank[op++] = r;
  r = 0;
  sp->n_in = op;
  for (const char* p = arrow + 2; *p; ++p) {
    int e = add(*p);
    if (e) return e;
  }
  if (r == 0) return fail(EA_ERR_SPEC, "spec '%s': empty output", s);
  sp->rank[op] = r;
  for (int i = 0; i < r; ++i) {
    bool found = false;
    for (int o = 0; o < sp->n_in && !found; ++o)
      for (int j = 0; j < sp->rank[o]; ++j) found |= sp->let[o][j] == sp->let[op][i];
    if (!found) return fail(EA_ERR_SPEC, "spec '%s': output letter '%c' in no input", s, sp->let[op][i]);
  }
  return EA_OK;
}

int find_dim(const Spec& sp, int op, char l) {
  for (int d = 0; d < sp.rank[op]; ++d)
    if (sp.let[op][d] == l) return d;
  return -1;
}
}  // namespace ea

namespace {

// ---------------------------------------------------------------------------
// join analysis: letter order, partitions, validation (Section 3.2)
// ---------------------------------------------------------------------------
struct JoinInfo {
  std::vector<char> letters;                  // group letters, then the rest
  int n_group = 0;
  std::vector<std::vector<int64_t>> lsplits;  // per letter: its split points
  std::vector<int64_t> lext;
  int index(char l) const {
    for (size_t i = 0; i < letters.size(); ++i)
      if (letters[i] == l) return (int)i;
    return -1;
  }
};

// ops: n_in inputs then the output.  group: output letters that key a group.
int analyze_join(const Spec& sp, const ea_relation* const* ops, const std::string& group, JoinInfo* ji) {
  const int n_ops = sp.n_in + 1;
  for (int o = 0; o < n_ops; ++o)
    if (ops[o]->rank != sp.rank[o])
      return fail(EA_ERR_SPEC, "operand %d has rank %d but the spec gives it %d letters", o, ops[o]->rank,
                  sp.rank[o]);
  *ji = JoinInfo();
  for (char l : group) ji->letters.push_back(l);
  ji->n_group = (int)group.size();
  for (int o = 0; o < sp.n_in; ++o)
    for (int d = 0; d < sp.rank[o]; ++d)
      if (ji->index(sp.let[o][d]) < 0) ji->letters.push_back(sp.let[o][d]);
  if ((int)ji->letters.size() > kMaxLetters) return fail(EA_ERR_UNSUPPORTED, "more than %d letters", kMaxLetters);
  ji->lsplits.assign(ji->letters.size(), {});
  ji->lext.assign(ji->letters.size(), 0);
  for (size_t li = 0; li < ji->letters.size(); ++li) {
    const char l = ji->letters[li];
    int first_op = -1;
    for (int o = 0; o < n_ops; ++o) {
      const int d = find_dim(sp, o, l);
      if (d < 0) continue;
      if (first_op < 0) {
        first_op = o;
        ji->lsplits[li] = ops[o]->splits[d];
        ji->lext[li] = ops[o]->shape[d];
        continue;
      }
      if (ops[o]->shape[d] != ji->lext[li])
        return fail(EA_ERR_SPEC, "letter '%c' has extent %lld in operand %d and %lld in operand %d", l,
                    (long long)ji->lext[li], first_op, (long long)ops[o]->shape[d], o);
      if (ops[o]->splits[d] != ji->lsplits[li]) {
        if (o == sp.n_in)
          return fail(EA_ERR_JOIN,
                      "output partition on letter '%c' differs from the inputs' (the output tiling "
                      "must be the one the join induces)", l);
        return fail(EA_ERR_JOIN,
                    "letter '%c' is split differently in operands %d and %d; repartition first", l,
                    first_op, o);
      }
    }
  }
  return EA_OK;
}

// ---------------------------------------------------------------------------
// plan image: host-built sections uploaded once into the plan's device buffer
// ---------------------------------------------------------------------------
struct Image {
  std::vector<uint8_t> bytes;
  size_t put(const void* p, size_t n) {
    size_t o = (size_t)align256((int64_t)bytes.size());
    bytes.resize(o + std::max<size_t>(n, 1), 0);
    if (n) memcpy(bytes.data() + o, p, n);
    return o;
  }
  size_t put_zero(size_t n) {
    size_t o = (size_t)align256((int64_t)bytes.size());
    bytes.resize(o + std::max<size_t>(n, 1), 0);
    return o;
  }
  template <class T>
  size_t put_vec(const std::vector<T>& v) { return put(v.data(), v.size() * sizeof(T)); }
};

enum Kind { K_GENERIC = 1, K_GEMM, K_GEMM32, K_RMSNORM, K_SOFTMAX, K_ATTENTION, K_REPART };

// row-reduction plan constants (see RowArgs)
struct RowLayout {
  int32_t row_len = 0, vec = 0, cps = 0, affine = 0, seg_len = 0, nseg = 0;
  int64_t xs = 0, ys = 0, ws = 0, wbase = 0;
};

struct Plan {
  int device = 0;
  Kind kind = K_GENERIC;
  char* dmem = nullptr;   // tables of the join and the work list
  size_t dbytes = 0;
  char* dmem2 = nullptr;  // attention: work units and their block records
  // join
  int n_in = 0;
  int64_t n_groups = 0, tuple_cap = 0;
  int32_t* d_tuples = nullptr;
  int32_t* d_goff = nullptr;
  int32_t* d_count = nullptr;
  const DevBlk* d_blk[kMaxOps] = {};
  // kernel-specific
  const void* d_desc = nullptr;
  const void* d_work = nullptr;
  int64_t n_work = 0;
  // gemm
  int b_kmajor = 0;
  int gemm_parts = 1;
  bool gemm_direct = false;  // direct-load kernel (work list of GemmUnit), else GemmTile
  int gemm_tn = kGemmTN;     // output tile columns per right operand (256, or 128)
  GemmTupleMeta* d_gemm_meta = nullptr;  // direct-load plans: per-tuple operand blocks
  // repartition: tasks of kRepTaskBytesSmall (relations below kRepLargeBytes)
  bool rep_small = false;
  // rows
  RowLayout rows;
  AttnUnitMeta* attn_meta = nullptr;
  // Caller workspace of split keys: arrival counters at the start of the
  // counter area, partial results after the area (attention: O partials,
  // then (m, l) partials at ws_part_ml).
  int64_t ws_counters = 0;
  int64_t ws_partial_bytes = 0;
  size_t ws_part_ml = 0;
  int64_t ws_bytes() const { return ws_counters || ws_partial_bytes ? kWsCounterBytes + ws_partial_bytes : 0; }
  ~Plan() {
    if (dmem || dmem2) {
      int cur = 0;
      if (hipGetDevice(&cur) == hipSuccess) {
        (void)hipSetDevice(device);
        (void)hipDeviceSynchronize();
        if (dmem) (void)hipFree(dmem);
        if (dmem2) (void)hipFree(dmem2);
        (void)hipSetDevice(cur);
      }
    }
  }
};

std::mutex g_cache_mu;
std::map<std::string, std::unique_ptr<Plan>>& cache() {
  static auto* m = new std::map<std::string, std::unique_ptr<Plan>>();  // intentionally leaked at exit
  return *m;
}

void key_rel(std::ostringstream& k, const ea_relation* r) {
  k << "|t" << r->dtype << "r" << r->rank;
  for (int d = 0; d < r->rank; ++d) {
    k << "[";
    for (int64_t s : r->splits[d]) k << s << ",";
    k << "]";
  }
}

// Allocate a device buffer for a plan image and upload the image into it.
int upload_image(const Image& img, char** mem, hipStream_t s) {
  EA_HIP_TRY(hipMalloc((void**)mem, std::max<size_t>(img.bytes.size(), 256)));
  EA_HIP_TRY(hipMemcpyAsync(*mem, img.bytes.data(), img.bytes.size(), hipMemcpyHostToDevice, s));
  return EA_OK;
}

int plan_upload(Plan* p, const Image& img, hipStream_t s) {
  p->dbytes = img.bytes.size();
  EA_HIP_TRY(hipGetDevice(&p->device));
  return upload_image(img, &p->dmem, s);
}

// Build the enumerator description and reserve the tuple table.
struct JoinSections {
  size_t desc, splits, tuples, goff, count;
  size_t blk[kMaxOps];
};

struct OpInfo {
  Kind kind = K_GENERIC;
  std::string group;   // group letters
  int causal = 0;      // the kernel masks keys after the query position
  int join_causal = 0; // the join drops tuples whose key block is fully masked
  char cq = 0, ck = 0; // causal letters
  int b_kmajor = 0;
  int q_dim = 0, k_dim = 0;
  int gqa = 1;                   // query heads per key/value head (attention)
  char gh = 0, gg = 0;           // query-head and key/value-head letters (gqa > 1)
  int head_dim = -1;             // their dim in Q and in K/V
  std::vector<int64_t> seq_ends; // packed sequences along cq/ck (attention), empty: one
};

int build_join(const Spec& sp, const ea_relation* const* ops, const JoinInfo& ji, const OpInfo& oi, Image* img,
               JoinSections* js, int64_t* n_groups, int64_t* tuple_cap) {
  const int causal = oi.join_causal;
  EnumDesc e;
  memset(&e, 0, sizeof(e));
  e.n_in = sp.n_in;
  e.n_letters = (int32_t)ji.letters.size();
  e.n_group_letters = ji.n_group;
  std::vector<int32_t> sp32;
  int64_t per_group = 1, ng = 1;
  for (size_t li = 0; li < ji.letters.size(); ++li) {
    e.letter_nb[li] = (int32_t)(ji.lsplits[li].size() - 1);
    e.letter_split[li] = (int32_t)sp32.size();
    for (int64_t v : ji.lsplits[li]) sp32.push_back((int32_t)v);
    if ((int)li < ji.n_group) ng *= e.letter_nb[li];
    else per_group *= e.letter_nb[li];
  }
  for (int o = 0; o <= sp.n_in; ++o) {
    e.op_rank[o] = sp.rank[o];
    for (int d = 0; d < sp.rank[o]; ++d) {
      e.op_letter[o][d] = ji.index(sp.let[o][d]);
      e.op_nb[o][d] = ops[o]->nb[d];
      e.op_split[o][d] = (int32_t)sp32.size();
      for (int64_t v : ops[o]->splits[d]) sp32.push_back((int32_t)v);
    }
  }
  e.causal = causal;
  if (causal || !oi.seq_ends.empty()) {
    e.cq = ji.index(oi.cq);
    e.ck = ji.index(oi.ck);
    if (e.cq < 0 || e.ck < 0) return fail(EA_ERR_SPEC, "query/key letters not in the spec");
  }
  if (oi.gqa > 1) {  // grouped-query heads
    e.gqa = oi.gqa;
    e.gh = ji.index(oi.gh);
    e.gg = ji.index(oi.gg);
    if (e.gh < 0 || e.gg < 0) return fail(EA_ERR_SPEC, "head letters not in the spec");
  }
  if (!oi.seq_ends.empty()) {  // packed sequences: their ends after the split lists
    e.n_seq = (int32_t)oi.seq_ends.size();
    e.seq_split = (int32_t)sp32.size();
    for (int64_t v : oi.seq_ends) sp32.push_back((int32_t)v);
  }
  e.per_group = per_group;
  e.n_groups = ng;
  e.n_cand = per_group * ng;
  if (e.n_cand > (int64_t)1 << 26) return fail(EA_ERR_UNSUPPORTED, "join space of %lld candidates is too large", (long long)e.n_cand);
  js->desc = img->put(&e, sizeof(e));
  js->splits = img->put_vec(sp32);
  js->tuples = img->put_zero((size_t)e.n_cand * (size_t)(sp.n_in + 1) * sizeof(int32_t));
  js->goff = img->put_zero((size_t)(ng + 1) * sizeof(int32_t));
  js->count = img->put_zero(sizeof(int32_t));
  for (int o = 0; o <= sp.n_in; ++o) js->blk[o] = img->put_vec(dev_blocks(ops[o]));
  *n_groups = ng;
  *tuple_cap = e.n_cand;
  return EA_OK;
}

int finish_join(Plan* p, const JoinSections& js, int n_ops, hipStream_t s) {
  p->d_tuples = (int32_t*)(p->dmem + js.tuples);
  p->d_goff = (int32_t*)(p->dmem + js.goff);
  p->d_count = (int32_t*)(p->dmem + js.count);
  for (int o = 0; o < n_ops; ++o) p->d_blk[o] = (const DevBlk*)(p->dmem + js.blk[o]);
  EA_HIP_TRY(launch_enumerate((const EnumDesc*)(p->dmem + js.desc), (const int32_t*)(p->dmem + js.splits),
                              p->d_tuples, p->d_goff, p->d_count, s));
  EA_HIP_TRY(hipStreamSynchronize(s));
  return EA_OK;
}

// ---------------------------------------------------------------------------
// operation classification and validation
// ---------------------------------------------------------------------------

// largest block of a relation, in bytes
int64_t max_block_bytes(const ea_relation* r) {
  int64_t n = dtype_size(r->dtype);
  for (int d = 0; d < r->rank; ++d) {
    int64_t m = 0;
    for (int b = 0; b < r->nb[d]; ++b) m = std::max<int64_t>(m, r->splits[d][b + 1] - r->splits[d][b]);
    n *= m;
  }
  return n;
}

bool is_float_dtype(int32_t dt) { return dt == EA_F32 || dt == EA_BF16 || dt == EA_F16; }

int classify(const Spec& sp, int32_t join_op, int32_t agg_op, const ea_relation* const* ops,
             const ea_params* prm, OpInfo* oi) {
  const int n_in = sp.n_in, out = n_in;
  const ea_relation* o = ops[out];
  std::string out_letters(sp.let[out], sp.let[out] + sp.rank[out]);
  *oi = OpInfo();
  for (int i = 0; i <= n_in; ++i)
    if (!is_float_dtype(ops[i]->dtype)) return fail(EA_ERR_DTYPE, "operand %d has an unknown dtype", i);
  switch (join_op) {
    case EA_JOIN_MUL:
    case EA_JOIN_ADD: {
      if (agg_op != EA_AGG_NONE && agg_op != EA_AGG_SUM && agg_op != EA_AGG_MAX)
        return fail(EA_ERR_ARG, "einsum joins aggregate with NONE, SUM or MAX");
      bool contracted = false;
      for (int i = 0; i < n_in; ++i)
        for (int d = 0; d < sp.rank[i]; ++d) contracted |= find_dim(sp, out, sp.let[i][d]) < 0;
      if (agg_op == EA_AGG_NONE && contracted)
        return fail(EA_ERR_SPEC, "aggregation NONE with contracted letters: several tuples share an output key");
      oi->group = out_letters;
      oi->kind = K_GENERIC;
      if (prm && prm->residual) {
        const ea_relation* r = prm->residual;
        if (r->rank != o->rank || r->dtype != o->dtype)
          return fail(EA_ERR_ARG, "residual relation must have the output's rank and dtype");
        for (int d = 0; d < o->rank; ++d)
          if (r->splits[d] != o->splits[d]) return fail(EA_ERR_ARG, "residual partition differs from the output's");
        if (!r->data) return fail(EA_ERR_ARG, "residual relation has no data");
      }
      // fp32 block products "ab,bc->ac" / "ab,cb->ac" without a residual:
      // the vector-ALU tile kernel
      if (join_op == EA_JOIN_MUL && agg_op == EA_AGG_SUM && n_in == 2 && sp.rank[0] == 2 && sp.rank[1] == 2 &&
          sp.rank[2] == 2 && ops[0]->dtype == EA_F32 && ops[1]->dtype == EA_F32 && !(prm && prm->residual)) {
        const char a = sp.let[0][0], b = sp.let[0][1];
        const char* L1 = sp.let[1];
        const char* L2 = sp.let[2];
        int kmaj = -1;
        char c = 0;
        if (L1[0] == b && L1[1] != a && L1[1] != b) { kmaj = 0; c = L1[1]; }
        else if (L1[1] == b && L1[0] != a && L1[0] != b) { kmaj = 1; c = L1[0]; }
        if (kmaj >= 0 && L2[0] == a && L2[1] == c) {
          oi->kind = K_GEMM32;
          oi->b_kmajor = kmaj;
          return EA_OK;
        }
      }
      // matrix-core path: "ab,bc->ac" or "ab,cb->ac", 16-bit inputs, SUM of products
      if (join_op == EA_JOIN_MUL && agg_op == EA_AGG_SUM && n_in == 2 && sp.rank[0] == 2 &&
          sp.rank[1] == 2 && sp.rank[2] == 2 && ops[0]->dtype == ops[1]->dtype &&
          (ops[0]->dtype == EA_BF16 || ops[0]->dtype == EA_F16)) {
        const char a = sp.let[0][0], b = sp.let[0][1];
        const char* L1 = sp.let[1];
        const char* L2 = sp.let[2];
        int kmaj = -1;
        char c = 0;
        if (L1[0] == b && L1[1] != a && L1[1] != b) { kmaj = 0; c = L1[1]; }
        else if (L1[1] == b && L1[0] != a && L1[0] != b) { kmaj = 1; c = L1[0]; }
        if (kmaj >= 0 && L2[0] == a && L2[1] == c) {
          // 16-byte vector loads and stores need 8-element-aligned block rows:
          // the contracted letter in both operands and the output columns
          bool aligned = true;
          for (int64_t v : ops[0]->splits[1]) aligned &= v % 8 == 0;
          for (int64_t v : ops[1]->splits[0]) aligned &= v % 8 == 0;
          for (int64_t v : ops[1]->splits[1]) aligned &= v % 8 == 0;
          if (aligned) {
            oi->kind = K_GEMM;
            oi->b_kmajor = kmaj;
          }
        }
      }
      return EA_OK;
    }
    case EA_OP_SWIGLU: {
      if (agg_op != EA_AGG_SUM) return fail(EA_ERR_ARG, "SWIGLU aggregates with SUM");
      if (n_in != 3 || sp.rank[0] != 2 || sp.rank[1] != 2 || sp.rank[2] != 2 || sp.rank[3] != 2)
        return fail(EA_ERR_SPEC, "SWIGLU spec must be 'tj,jk,jk->tk' (or 'tj,kj,kj->tk')");
      const char t = sp.let[0][0], j = sp.let[0][1];
      int kmaj = -1;
      char k = 0;
      if (sp.let[1][0] == j) { kmaj = 0; k = sp.let[1][1]; }
      else if (sp.let[1][1] == j) { kmaj = 1; k = sp.let[1][0]; }
      if (kmaj < 0 || k == t || k == j || sp.let[2][0] != sp.let[1][0] || sp.let[2][1] != sp.let[1][1] ||
          sp.let[3][0] != t || sp.let[3][1] != k)
        return fail(EA_ERR_SPEC, "SWIGLU spec must be 'tj,jk,jk->tk' (or 'tj,kj,kj->tk')");
      for (int i = 0; i < 3; ++i)
        if (ops[i]->dtype != EA_BF16 && ops[i]->dtype != EA_F16)
          return fail(EA_ERR_DTYPE, "SWIGLU takes bf16 or f16 inputs");
      if (ops[1]->dtype != ops[0]->dtype || ops[2]->dtype != ops[0]->dtype)
        return fail(EA_ERR_DTYPE, "SWIGLU inputs must share one dtype");
      for (int64_t v : ops[0]->splits[1])
        if (v % 8) return fail(EA_ERR_UNSUPPORTED, "SWIGLU needs contracted block bounds that are multiples of 8");
      for (int64_t v : ops[1]->splits[1])
        if (v % 8) return fail(EA_ERR_UNSUPPORTED, "SWIGLU needs weight block bounds that are multiples of 8");
      if (prm && prm->residual) return fail(EA_ERR_UNSUPPORTED, "SWIGLU takes no residual");
      oi->kind = K_GEMM;
      oi->b_kmajor = kmaj;
      oi->group = out_letters;
      return EA_OK;
    }
    case EA_OP_RMSNORM: {
      if (agg_op != EA_AGG_SUM) return fail(EA_ERR_ARG, "RMSNORM aggregates its sum of squares with SUM");
      if (n_in != 2 || sp.rank[1] != 1 || sp.rank[out] != sp.rank[0])
        return fail(EA_ERR_SPEC, "RMSNORM spec must be '<r>c,c-><r>c'");
      const char c = sp.let[0][sp.rank[0] - 1];
      if (sp.let[1][0] != c || out_letters != std::string(sp.let[0], sp.let[0] + sp.rank[0]))
        return fail(EA_ERR_SPEC, "RMSNORM spec must be '<r>c,c-><r>c'");
      if (!prm || !(prm->eps >= 0.0f)) return fail(EA_ERR_ARG, "RMSNORM needs params with eps >= 0");
      if (ops[0]->dtype == EA_F16 || ops[1]->dtype == EA_F16 || o->dtype == EA_F16)
        return fail(EA_ERR_DTYPE, "RMSNORM takes f32 or bf16");
      if (prm->residual) return fail(EA_ERR_UNSUPPORTED, "RMSNORM takes no residual");
      oi->kind = K_RMSNORM;
      oi->group = out_letters.substr(0, out_letters.size() - 1);
      return EA_OK;
    }
    case EA_OP_SOFTMAX: {
      if (agg_op != EA_AGG_LSE) return fail(EA_ERR_ARG, "SOFTMAX aggregates with LSE (max, then sum)");
      if (n_in != 1 || out_letters != std::string(sp.let[0], sp.let[0] + sp.rank[0]))
        return fail(EA_ERR_SPEC, "SOFTMAX spec must be 'X->X'");
      if (ops[0]->dtype == EA_F16 || o->dtype == EA_F16) return fail(EA_ERR_DTYPE, "SOFTMAX takes f32 or bf16");
      const int causal = prm ? prm->causal : 0;
      if (causal && sp.rank[0] < 2) return fail(EA_ERR_SPEC, "causal SOFTMAX needs a query letter");
      if (prm && prm->residual) return fail(EA_ERR_UNSUPPORTED, "SOFTMAX takes no residual");
      // Masked entries of a softmax are stored zeros of the output, so its
      // join keeps every key block; the kernel applies the mask per element.
      oi->kind = K_SOFTMAX;
      oi->group = out_letters.substr(0, out_letters.size() - 1);
      oi->causal = causal;
      return EA_OK;
    }
    case EA_OP_ATTENTION: {
      if (agg_op != EA_AGG_LSE) return fail(EA_ERR_ARG, "ATTENTION aggregates with LSE (online softmax)");
      if (n_in != 3) return fail(EA_ERR_SPEC, "ATTENTION spec must be '<b>qd,<b>kd,<b>kd-><b>qd'");
      const int r = sp.rank[0];
      const int gqa = prm && prm->gqa_group > 1 ? prm->gqa_group : 1;
      bool good = r >= 2 && sp.rank[1] == r && sp.rank[2] == r && sp.rank[out] == r;
      char q = 0, k = 0, d = 0;
      int hd = -1;  // grouped-query: the batch dim where K/V name their own head letter
      if (good) {
        q = sp.let[0][r - 2];
        d = sp.let[0][r - 1];
        k = sp.let[1][r - 2];
        good = k != q && k != d && sp.let[1][r - 1] == d && sp.let[2][r - 2] == k && sp.let[2][r - 1] == d;
        for (int i = 0; i < r - 2 && good; ++i) {
          good = sp.let[2][i] == sp.let[1][i];
          if (sp.let[1][i] == sp.let[0][i]) continue;
          // a K/V letter apart from Q's: only the one head letter of GQA
          good = good && gqa > 1 && hd < 0 && find_dim(sp, 0, sp.let[1][i]) < 0;
          hd = i;
        }
        good = good && out_letters == std::string(sp.let[0], sp.let[0] + r);
      }
      if (!good)
        return fail(EA_ERR_SPEC, gqa > 1 ? "grouped-query ATTENTION spec must be '<b>hqd,<b>gkd,<b>gkd-><b>hqd'"
                                         : "ATTENTION spec must be '<b>qd,<b>kd,<b>kd-><b>qd'");
      if (gqa > 1) {
        if (hd < 0) return fail(EA_ERR_SPEC, "grouped-query ATTENTION needs a key/value head letter apart from Q's");
        if (ops[0]->shape[hd] != (int64_t)gqa * ops[1]->shape[hd])
          return fail(EA_ERR_SPEC, "grouped-query ATTENTION: %lld query heads are not %d x %lld key/value heads",
                      (long long)ops[0]->shape[hd], gqa, (long long)ops[1]->shape[hd]);
        if (ops[1]->nb[hd] != ops[1]->shape[hd])
          return fail(EA_ERR_UNSUPPORTED, "ATTENTION needs one block per key/value head");
      }
      for (int i = 0; i < 3; ++i)
        if (ops[i]->dtype != EA_BF16) return fail(EA_ERR_DTYPE, "ATTENTION takes bf16 Q, K, V");
      if (o->dtype == EA_F16) return fail(EA_ERR_DTYPE, "ATTENTION writes f32 or bf16");
      if (ops[0]->shape[r - 1] != 128 || ops[0]->nb[r - 1] != 1)
        return fail(EA_ERR_UNSUPPORTED, "ATTENTION needs head dim 128 in one block");
      for (int64_t v : ops[0]->splits[r - 2])
        if (v % 128) return fail(EA_ERR_UNSUPPORTED, "ATTENTION needs query block bounds that are multiples of 128");
      for (int64_t v : ops[1]->splits[r - 2])
        if (v % 128) return fail(EA_ERR_UNSUPPORTED, "ATTENTION needs key block bounds that are multiples of 128");
      for (int dd = 0; dd < r - 2; ++dd)
        if (ops[0]->nb[dd] != ops[0]->shape[dd])
          return fail(EA_ERR_UNSUPPORTED, "ATTENTION needs one block per batch-letter index (dim %d)", dd);
      const int causal = prm ? prm->causal : 0;
      if (causal && ops[0]->shape[r - 2] != ops[1]->shape[r - 2])
        return fail(EA_ERR_SPEC, "causal ATTENTION needs as many queries as keys");
      if (!prm || !(std::isfinite(prm->scale)) || !(prm->scale > 0.0f))
        return fail(EA_ERR_ARG, "ATTENTION needs params with a positive finite scale");
      if (prm->residual) return fail(EA_ERR_UNSUPPORTED, "ATTENTION takes no residual");
      if (prm->n_seq < 0 || (prm->n_seq > 0 && !prm->seq_ends))
        return fail(EA_ERR_ARG, "ATTENTION: n_seq %d with seq_ends %p", prm->n_seq, (const void*)prm->seq_ends);
      if (prm->n_seq > 0) {
        // packed sequences: strictly increasing ends, the last the extent,
        // each a split point of the query and of the key partition
        const int64_t S = ops[0]->shape[r - 2];
        if (ops[1]->shape[r - 2] != S) return fail(EA_ERR_SPEC, "packed-sequence ATTENTION needs as many queries as keys");
        if (prm->n_seq > (1 << 20)) return fail(EA_ERR_ARG, "ATTENTION: %d sequences", prm->n_seq);
        int64_t prev = 0;
        for (int i = 0; i < prm->n_seq; ++i) {
          const int64_t e = prm->seq_ends[i];
          if (e <= prev || e > S) return fail(EA_ERR_ARG, "ATTENTION: sequence end %d (%lld) out of order", i, (long long)e);
          for (int op = 0; op < 2; ++op) {
            const std::vector<int64_t>& ss = ops[op]->splits[r - 2];
            if (!std::binary_search(ss.begin(), ss.end(), e))
              return fail(EA_ERR_UNSUPPORTED, "ATTENTION: sequence end %lld is not a %s block bound", (long long)e,
                          op ? "key" : "query");
          }
          prev = e;
        }
        if (prev != S) return fail(EA_ERR_ARG, "ATTENTION: the last sequence end %lld is not the extent %lld",
                                   (long long)prev, (long long)S);
        oi->seq_ends.assign(prm->seq_ends, prm->seq_ends + prm->n_seq);
      }
      // A fully masked key block contributes nothing to O: the join drops it.
      oi->kind = K_ATTENTION;
      oi->group = out_letters;
      oi->causal = causal;
      oi->join_causal = causal;
      oi->cq = q;
      oi->ck = k;
      oi->q_dim = r - 2;
      oi->k_dim = r - 2;
      if (gqa > 1) {
        oi->gqa = gqa;
        oi->gh = sp.let[0][hd];
        oi->gg = sp.let[1][hd];
        oi->head_dim = hd;
      }
      return EA_OK;
    }
    default:
      return fail(EA_ERR_ARG, "unknown join op %d", join_op);
  }
}

// ---------------------------------------------------------------------------
// kind-specific plan sections
// ---------------------------------------------------------------------------
struct Extra {
  size_t desc = 0, work = 0, meta = 0;
  int64_t n_work = 0;
};

int build_generic(const Spec& sp, int32_t join_op, int32_t agg_op, const ea_relation* const* ops,
                  const JoinInfo& ji, const ea_relation* res, Image* img, Extra* ex) {
  GenDesc g;
  memset(&g, 0, sizeof(g));
  const int out = sp.n_in;
  g.n_in = sp.n_in;
  g.join = join_op;
  g.agg = agg_op;
  g.has_res = res != nullptr;
  g.out_rank = sp.rank[out];
  g.dt_out = ops[out]->dtype;
  g.dt_res = res ? res->dtype : 0;
  for (int d = 0; d < sp.rank[out]; ++d) g.out_letter[d] = ji.index(sp.let[out][d]);
  for (int i = 0; i < sp.n_in; ++i) {
    g.in_rank[i] = sp.rank[i];
    g.dt_in[i] = ops[i]->dtype;
    for (int d = 0; d < sp.rank[i]; ++d) g.in_letter[i][d] = ji.index(sp.let[i][d]);
  }
  for (size_t li = 0; li < ji.letters.size(); ++li) {
    if (find_dim(sp, out, ji.letters[li]) >= 0) continue;
    for (int i = 0; i < sp.n_in; ++i) {
      int d = find_dim(sp, i, ji.letters[li]);
      if (d >= 0) {
        g.contr_letter[g.n_contr] = (int32_t)li;
        g.contr_op[g.n_contr] = i;
        g.contr_dim[g.n_contr] = d;
        ++g.n_contr;
        break;
      }
    }
  }
  std::vector<GenWork> work;
  const ea_relation* o = ops[out];
  for (int64_t b = 0; b < o->nblocks; ++b) {
    int64_t n = 1;
    int32_t c[kMaxRank];
    block_coords(o, b, c);
    for (int d = 0; d < o->rank; ++d) n *= o->splits[d][c[d] + 1] - o->splits[d][c[d]];
    if (n > INT32_MAX) return fail(EA_ERR_UNSUPPORTED, "output block too large for the generic kernel");
    for (int64_t s = 0; s < n; s += 256) work.push_back(GenWork{(int32_t)b, (int32_t)s});
  }
  ex->desc = img->put(&g, sizeof(g));
  ex->work = img->put_vec(work);
  ex->n_work = (int64_t)work.size();
  return EA_OK;
}

// Work units of a block-GEMM plan: every output block is cut into tiles of
// kGemmTM x tn; a tile whose group has many tuples may be split into n_parts
// runs of tuples (the SUM over the runs is merged by the kernel).  The split
// count minimises a simple time model on 256 CUs (one workgroup per CU):
//   waves(units) * ceil(iterations / parts) * t_step + merge traffic / BW
// with t_step ~ 1 us per 64-deep K step of a full tile and the merge writing
// and reading one 256 KiB fp32 partial per unit at ~4 TB/s.
// Units are then ordered so that the workgroups one XCD receives (ids
// congruent mod 8) form a compact rectangle of the tile grid and share
// operand panels in that XCD's L2.
// K-step time of a 256 x 128 tile over that of a 256 x 256 one.  Measured on
// the block share's QKV projection (2048 x 8192 x 3072), 192 workgroups
// either way: 256 x 128 tiles, 256 K steps each, 142.6 us; 256 x 256 tiles
// split in two, 128 K steps each plus the merge, 107.8 us (about 15 us of it
// the merge): 0.557 against 0.725 us per step.
constexpr double kNarrowStep = 0.77;

struct GemmPlanInfo {
  std::vector<GemmTile> units;
  int32_t slots = 0, counters = 0;
  int parts = 1;
};

GemmPlanInfo gemm_units(const ea_relation* a, const ea_relation* c, int tn, double step_scale = 1.0) {
  const int kCUs = 256;
  const double tile_bytes = (double)kGemmTM * tn * 4;
  // K steps of a group: every group has the same contracted blocks (a's column blocks)
  int64_t steps = 0;
  const int n_t = a->nb[1];
  for (int b = 0; b < n_t; ++b) steps += (a->splits[1][b + 1] - a->splits[1][b] + 63) / 64;
  std::vector<GemmTile> nat;
  int32_t co[kMaxRank];
  for (int64_t b = 0; b < c->nblocks; ++b) {
    block_coords(c, b, co);
    const int64_t me = c->splits[0][co[0] + 1] - c->splits[0][co[0]];
    const int64_t ne = c->splits[1][co[1] + 1] - c->splits[1][co[1]];
    for (int64_t m0 = 0; m0 < me; m0 += kGemmTM)
      for (int64_t n0 = 0; n0 < ne; n0 += tn) {
        GemmTile t;
        memset(&t, 0, sizeof(t));
        t.block = (int32_t)b;
        t.m0 = (int32_t)m0;
        t.n0 = (int32_t)n0;
        t.n_parts = 1;
        t.slot = t.first_slot = t.counter = -1;
        nat.push_back(t);
      }
  }
  const int64_t tiles = (int64_t)nat.size();
  int best_p = 1;
  double best_t = 1e300;
  for (int P = 1; P <= std::min(n_t, 16); ++P) {
    const int64_t units = tiles * P;
    const double waves = (double)((units + kCUs - 1) / kCUs);
    const double t = waves * (double)((steps + P - 1) / P) * step_scale + (P > 1 ? units * 2.0 * tile_bytes / 4.0e6 : 0.0);
    if (t < best_t - 1e-9) {
      best_t = t;
      best_p = P;
    }
  }
  GemmPlanInfo info;
  info.parts = best_p;
  std::vector<GemmTile> all;
  for (const GemmTile& t0 : nat) {
    for (int p = 0; p < best_p; ++p) {
      GemmTile t = t0;
      t.part = p;
      t.n_parts = best_p;
      if (best_p > 1) {
        t.slot = info.slots + p;
        t.first_slot = info.slots;
        t.counter = info.counters;
      }
      all.push_back(t);
    }
    if (best_p > 1) {  // the next tile's slots and counter
      info.slots += best_p;
      info.counters += 1;
    }
  }
  // XCD-aware order.  Workgroup i runs on XCD i % 8, and the eight XCDs have
  // private L2 caches, so each XCD gets a compact rectangle of the tile grid
  // (global tile rows mi x tile columns ni) of one part: its workgroups then
  // share the fewest distinct A row panels and B column panels at every K
  // step.  With P parts and P dividing 8, each part has 8 / P XCDs; else
  // every part is spread over all eight.
  std::vector<int> mrow(c->nb[0] + 1, 0), ncol(c->nb[1] + 1, 0);
  for (int b = 0; b < c->nb[0]; ++b)
    mrow[b + 1] = mrow[b] + (int)((c->splits[0][b + 1] - c->splits[0][b] + kGemmTM - 1) / kGemmTM);
  for (int b = 0; b < c->nb[1]; ++b) ncol[b + 1] = ncol[b] + (int)((c->splits[1][b + 1] - c->splits[1][b] + tn - 1) / tn);
  const int mt = mrow.back(), ntl = ncol.back();
  const int nx = 8;
  const bool split_parts = 8 % best_p == 0;
  const int per_part = split_parts ? 8 / best_p : 8;
  int gr = 1, gc = per_part;
  double best_perim = 1e300;
  for (int r = 1; r <= per_part; ++r) {
    if (per_part % r) continue;
    const int cc = per_part / r;
    const double perim = (double)mt / r + (double)ntl / cc + (r > mt ? 1e6 : 0) + (cc > ntl ? 1e6 : 0);
    if (perim < best_perim) {
      best_perim = perim;
      gr = r;
      gc = cc;
    }
  }
  struct Keyed {
    int64_t key;
    GemmTile t;
  };
  std::vector<std::vector<Keyed>> q(nx);
  for (const GemmTile& t : all) {
    block_coords(c, t.block, co);
    const int mi = mrow[co[0]] + t.m0 / kGemmTM, ni = ncol[co[1]] + t.n0 / tn;
    const int rb = (int)((int64_t)mi * gr / std::max(mt, 1)), cb = (int)((int64_t)ni * gc / std::max(ntl, 1));
    const int region = rb * gc + cb;
    const int x = split_parts ? (t.part * per_part + region) % nx : region % nx;
    // inside a region: part, then 4-row stripes walked column by column
    const int64_t key = (((int64_t)t.part * (mt / 4 + 1) + mi / 4) * (ntl + 1) + ni) * 4 + mi % 4;
    q[x].push_back(Keyed{key, t});
  }
  for (auto& v : q) std::stable_sort(v.begin(), v.end(), [](const Keyed& x, const Keyed& y) { return x.key < y.key; });
  const size_t n = all.size();
  std::vector<size_t> head(nx, 0);
  info.units.reserve(n);
  for (size_t p = 0; info.units.size() < n; ++p) {
    const size_t x = p % nx;
    if (head[x] < q[x].size()) {
      info.units.push_back(q[x][head[x]++].t);
      continue;
    }
    size_t y_best = nx;  // this XCD has run out: take from the fullest queue
    for (size_t y = 0; y < (size_t)nx; ++y)
      if (head[y] < q[y].size() && (y_best == nx || q[y].size() - head[y] > q[y_best].size() - head[y_best])) y_best = y;
    info.units.push_back(q[y_best][head[y_best]++].t);
  }
  return info;
}

// Units of the direct-load kernel (contracted block extents multiples of 32,
// at most kGemmMaxTuples tuples per group).  Two schedules are costed and the
// cheaper one is kept:
//   * even: the tiles of gemm_units (split or not, in XCD-aware order), one
//     segment each;
//   * balanced: the tiles' 32-deep K steps laid end to end (tiles in block
//     order) and cut into 256 equal runs, one per CU; a run may end one tile
//     and start the next, and a tile cut into several runs is merged by its
//     last arriver.  This fills every CU when there are fewer tiles than CUs.
// Time model (us): 0.75 per K step of a tile, 1 per segment (pipeline fill and
// store), and the split tiles' partial sums written and read back at an
// effective 8 TB/s: two-part tiles move two partials (the first arriver's
// write, the second's read), more parts every part's write and a read of
// each.  The rate is above HBM's because those exchanges partly overlap
// other workgroups' K steps; it is fitted to the block share, where balanced
// SwiGLU (176 tiles, 176 steps per run, almost every tile in two or three
// runs) measured 188 us against 191-194 us even, and balanced QKV 125 us
// against 109-112 us even.
// The step time grows once more than about 190 CUs run matrix work at once:
// the sustained clock is power-limited, so a schedule that keeps all 256 CUs
// busy gains less than its CU count suggests.
struct GemmDlPlan {
  std::vector<GemmUnit> units;
  int32_t slots = 0, counters = 0;
  bool balanced = false;
  double cost = 0.0;  // the model's time of the kept schedule (us)
};

GemmDlPlan gemm_units_dl(const ea_relation* a, const ea_relation* c, int tn, const GemmPlanInfo& even,
                         double step_scale = 1.0) {
  const int kCUs = 256;
  const double t_step = 0.75 * step_scale, t_seg = 1.0, bw = 8.0e6, tile_bytes = (double)kGemmTM * tn * 4,
               n_sat = 190.0;
  auto step_time = [&](int64_t busy_cus) { return t_step * std::max(1.0, (double)busy_cus / n_sat); };
  // K-step prefix over a group's tuples (A's contracted blocks, in order)
  const int n_t = a->nb[1];
  std::vector<int32_t> pre(n_t + 1, 0);
  for (int b = 0; b < n_t; ++b) pre[b + 1] = pre[b] + (int32_t)((a->splits[1][b + 1] - a->splits[1][b]) / 32);
  const int64_t S = pre[n_t];
  auto merge_bytes = [&](int parts) { return parts > 1 ? (parts == 2 ? 2 : 2 * parts) * tile_bytes : 0.0; };
  // even schedule, as one-segment units
  GemmDlPlan ev;
  double ev_cost = 0.0;
  {
    int64_t max_steps = 0;
    double bytes = 0.0;
    for (const GemmTile& t : even.units) {
      GemmUnit u;
      memset(&u, 0, sizeof(u));
      GemmSeg& g = u.seg[0];
      g.block = t.block;
      g.m0 = t.m0;
      g.n0 = t.n0;
      g.s0 = pre[(int)(((int64_t)t.part * n_t) / t.n_parts)];
      g.s1 = pre[(int)(((int64_t)(t.part + 1) * n_t) / t.n_parts)];
      g.part = t.part;
      g.n_parts = t.n_parts;
      g.first_slot = t.first_slot;
      g.counter = t.counter;
      u.n_seg = 1;
      ev.units.push_back(u);
      max_steps = std::max<int64_t>(max_steps, g.s1 - g.s0);
      if (t.part == 0) bytes += merge_bytes(t.n_parts);
    }
    ev.slots = even.slots;
    ev.counters = even.counters;
    const int64_t n_units = (int64_t)ev.units.size(), waves = (n_units + kCUs - 1) / kCUs;
    ev_cost = (double)waves * ((double)max_steps * step_time(std::min<int64_t>(n_units, kCUs)) + t_seg) + bytes / bw;
  }
  // balanced schedule
  std::vector<GemmTile> tiles;  // block order
  {
    int32_t co[kMaxRank];
    for (int64_t b = 0; b < c->nblocks; ++b) {
      block_coords(c, b, co);
      const int64_t me = c->splits[0][co[0] + 1] - c->splits[0][co[0]];
      const int64_t ne = c->splits[1][co[1] + 1] - c->splits[1][co[1]];
      for (int64_t m0 = 0; m0 < me; m0 += kGemmTM)
        for (int64_t n0 = 0; n0 < ne; n0 += tn) {
          GemmTile t;
          memset(&t, 0, sizeof(t));
          t.block = (int32_t)b;
          t.m0 = (int32_t)m0;
          t.n0 = (int32_t)n0;
          tiles.push_back(t);
        }
    }
  }
  ev.cost = ev_cost;
  const int64_t T = (int64_t)tiles.size(), total = T * S;
  if (T == 0 || S == 0 || T >= kCUs) return ev;  // a full wave of tiles: nothing to balance
  const int64_t q = (total + kCUs - 1) / kCUs;    // steps per unit (< S: at most two tiles per unit)
  if (q < 8) return ev;                           // too little work per unit to share
  GemmDlPlan bal;
  bal.balanced = true;
  std::vector<std::vector<std::pair<int, int>>> segs_of(T);  // (unit, seg) per tile, ascending s0
  for (int64_t u0 = 0; u0 < total; u0 += q) {
    GemmUnit u;
    memset(&u, 0, sizeof(u));
    const int64_t u1 = std::min(total, u0 + q);
    for (int64_t x = u0; x < u1;) {
      const int64_t t = x / S, e = std::min(u1, (t + 1) * S);
      if (u.n_seg >= kGemmMaxSegs) return ev;  // (cannot happen while q <= S)
      GemmSeg& g = u.seg[u.n_seg];
      g.block = tiles[(size_t)t].block;
      g.m0 = tiles[(size_t)t].m0;
      g.n0 = tiles[(size_t)t].n0;
      g.s0 = (int32_t)(x - t * S);
      g.s1 = (int32_t)(e - t * S);
      segs_of[(size_t)t].push_back({(int)bal.units.size(), u.n_seg});
      ++u.n_seg;
      x = e;
    }
    bal.units.push_back(u);
  }
  double bytes = 0.0;
  for (int64_t t = 0; t < T; ++t) {
    const auto& v = segs_of[(size_t)t];
    const int parts = (int)v.size();
    for (int i = 0; i < parts; ++i) {
      GemmSeg& g = bal.units[(size_t)v[i].first].seg[v[i].second];
      g.part = i;
      g.n_parts = parts;
      g.first_slot = parts > 1 ? bal.slots : -1;
      g.counter = parts > 1 ? bal.counters : -1;
    }
    if (parts > 1) {
      bal.slots += parts;
      bal.counters += 1;
    }
    bytes += merge_bytes(parts);
  }
  const double bal_cost = (double)q * step_time((int64_t)bal.units.size()) + 2.0 * t_seg + bytes / bw;
  bal.cost = bal_cost;
  // EA_GEMM_SCHEDULE=even|balanced overrides the model when a plan is built
  const char* force = getenv("EA_GEMM_SCHEDULE");
  if (force && !strcmp(force, "even")) return ev;
  if (force && !strcmp(force, "balanced")) return bal;
  return bal_cost < ev_cost ? bal : ev;
}

int build_rows(const Spec& sp, const ea_relation* const* ops, const OpInfo& oi, Image* img, Extra* ex,
               RowLayout* lay) {
  // rows of a group: points of the group letters' box; every group has the
  // same structure as block (g) of the output restricted to the group letters.
  const ea_relation* y = ops[sp.n_in];
  const ea_relation* x = ops[0];
  const ea_relation* w = oi.kind == K_RMSNORM ? ops[1] : nullptr;
  const int r = y->rank, dl = r - 1;
  const int es = dtype_size(x->dtype), esy = dtype_size(y->dtype);
  lay->row_len = (int32_t)y->shape[dl];
  bool aligned = true;
  for (int b = 0; b < x->nb[dl]; ++b) aligned &= (x->splits[dl][b + 1] - x->splits[dl][b]) * es % 16 == 0;
  lay->vec = rows_vec_ok(y->shape[dl], x->nb[dl], aligned, es) ? 1 : 0;
  // even segments (all but the last of one chunk count, the last no longer)
  const int64_t first = (x->splits[dl][1] - x->splits[dl][0]) * es / 16;
  bool even = aligned;
  for (int b = 0; b < x->nb[dl]; ++b) {
    const int64_t n = (x->splits[dl][b + 1] - x->splits[dl][b]) * es / 16;
    even &= b + 1 < x->nb[dl] ? n == first : n <= first;
  }
  lay->cps = even ? (int32_t)first : 0;
  // affine layout: equal segments, x and y with one partition (w along the
  // normalised letter too), and block offsets at fixed strides along it
  const int nseg = x->nb[dl];
  const int64_t L = x->splits[dl][1] - x->splits[dl][0];
  bool aff = lay->vec && even && x->rank == r;
  for (int b = 0; aff && b < nseg; ++b) aff &= x->splits[dl][b + 1] - x->splits[dl][b] == L;
  for (int d = 0; aff && d < r; ++d) aff &= x->splits[d] == y->splits[d];
  if (aff && w) aff &= w->rank == 1 && w->splits[0] == x->splits[dl];
  const int64_t xs = nseg > 1 ? x->off[1] - x->off[0] : 0, ys = nseg > 1 ? y->off[1] - y->off[0] : 0;
  const int64_t ws = w && nseg > 1 ? w->off[1] - w->off[0] : 0;
  for (int64_t b = 0; aff && b < x->nblocks; ++b) {
    const int64_t g = b / nseg, sg = b % nseg;
    aff &= x->off[b] == x->off[g * nseg] + sg * xs && y->off[b] == y->off[g * nseg] + sg * ys;
  }
  for (int sg = 0; aff && w && sg < nseg; ++sg) aff &= w->off[sg] == w->off[0] + sg * ws;
  lay->affine = aff ? 1 : 0;
  lay->seg_len = (int32_t)L;
  lay->nseg = nseg;
  lay->xs = xs;
  lay->ys = ys;
  lay->ws = ws;
  lay->wbase = w ? w->off[0] : 0;

  std::vector<RowTask> tasks;
  // groups enumerate block coordinates of the first r-1 dims, row-major
  int64_t n_groups = 1;
  for (int d = 0; d < r - 1; ++d) n_groups *= y->nb[d];
  int32_t c[kMaxRank] = {};
  const int rows_per_task = kRowsPerTask;  // the row kernels' wavefronts per workgroup
  const int qd = r - 2;
  for (int64_t g = 0; g < n_groups; ++g) {
    int64_t rem = g;
    for (int d = r - 2; d >= 0; --d) { c[d] = (int32_t)(rem % y->nb[d]); rem /= y->nb[d]; }
    int64_t rows = 1;
    for (int d = 0; d < r - 1; ++d) rows *= y->splits[d][c[d] + 1] - y->splits[d][c[d]];
    for (int64_t r0 = 0; r0 < rows; r0 += rows_per_task) {
      RowTask t;
      memset(&t, 0, sizeof(t));
      t.g = (int32_t)g;
      t.row0 = (int32_t)r0;
      t.nrows = (int32_t)std::min<int64_t>(rows_per_task, rows - r0);
      if (qd >= 0) {
        t.qlo = (int32_t)y->splits[qd][c[qd]];
        t.qext = (int32_t)(y->splits[qd][c[qd] + 1] - y->splits[qd][c[qd]]);
      }
      if (aff) {
        t.xrow = x->off[g * nseg] + r0 * L * es;
        t.yrow = y->off[g * nseg] + r0 * L * esy;
      }
      tasks.push_back(t);
    }
  }
  // causal softmax: a row's loads grow with its query position, so the
  // longest rows go first and the shortest fill the tail
  if (oi.kind == K_SOFTMAX && oi.causal && qd >= 0)
    std::stable_sort(tasks.begin(), tasks.end(), [](const RowTask& a, const RowTask& b) {
      return (int64_t)a.qlo + a.row0 % std::max(a.qext, 1) > (int64_t)b.qlo + b.row0 % std::max(b.qext, 1);
    });
  ex->work = img->put_vec(tasks);
  ex->n_work = (int64_t)tasks.size();
  return EA_OK;
}

// Work units of an attention plan.  Per group (b.., q block) and per 128-row
// query tile, the group's tuples (the key blocks the GPU join kept) are split
// into runs of at most kAttnMaxUnitTuples; the last unit of a split tile to
// finish merges the partials.  Tuple counts come from the GPU-built group
// offsets (goff), so the units follow the join's own predicates.
struct AttnPlanInfo {
  std::vector<AttnUnit> units;
  int32_t slots = 0, counters = 0;
};

int attention_units(const ea_relation* Q, const std::vector<int32_t>& goff, AttnPlanInfo* info) {
  const int r = Q->rank;
  const int64_t n_groups = Q->nblocks;  // group letters are all of Q's letters; d is one block
  if ((int64_t)goff.size() != n_groups + 1) return fail(EA_ERR_HIP, "internal: attention group count mismatch");
  struct TileWork {
    int64_t g, q0;
    int n_t;
  };
  std::vector<TileWork> tiles;
  int32_t c[kMaxRank];
  for (int64_t g = 0; g < n_groups; ++g) {
    block_coords(Q, g, c);
    const int64_t q_ext = Q->splits[r - 2][c[r - 2] + 1] - Q->splits[r - 2][c[r - 2]];
    const int n_t = goff[(size_t)g + 1] - goff[(size_t)g];
    if (n_t < 0) return fail(EA_ERR_HIP, "internal: GPU join group offsets decrease at group %lld", (long long)g);
    for (int64_t q0 = 0; q0 < q_ext; q0 += 128) tiles.push_back(TileWork{g, q0, n_t});
  }
  // key blocks per unit (the online-softmax partial): the run that minimises
  // waves of units over the 512 workgroup slots (two per CU) x (longest
  // unit + half a key block per extra part of a split tile, the merge); ties
  // go to the longer run
  const int kCUs = 512;
  int max_nt = 1;
  for (const TileWork& t : tiles) max_nt = std::max(max_nt, t.n_t);
  int chunk = kAttnMaxUnitTuples;
  double best = 1e300;
  for (int cc = kAttnMaxUnitTuples; cc >= 1; --cc) {
    int64_t n_units = 0;
    int max_parts = 1;
    for (const TileWork& t : tiles) {
      const int parts = std::max(1, (t.n_t + cc - 1) / cc);
      n_units += parts;
      max_parts = std::max(max_parts, parts);
    }
    const double waves = (double)((n_units + kCUs - 1) / kCUs);
    const double cost = waves * (std::min(cc, max_nt) + 0.5 * (max_parts - 1));
    if (cost < best - 1e-9) {
      best = cost;
      chunk = cc;
    }
  }
  int32_t slot = 0, counter = 0;
  for (const TileWork& t : tiles) {
    const int parts = std::max(1, (t.n_t + chunk - 1) / chunk);
    for (int p = 0; p < parts; ++p) {
      AttnUnit u;
      u.group = (int32_t)t.g;
      u.q0 = (int32_t)t.q0;
      u.part = p;
      u.n_parts = parts;
      u.weight = (t.n_t * (p + 1)) / parts - (t.n_t * p) / parts;
      if (u.weight > kAttnMaxUnitTuples)
        return fail(EA_ERR_HIP, "internal: attention unit of %d key blocks exceeds %d", u.weight, kAttnMaxUnitTuples);
      if (parts > 1) {
        u.slot = slot + p;
        u.first_slot = slot;
        u.counter = counter;
      } else {
        u.slot = -1;
        u.first_slot = -1;
        u.counter = -1;
      }
      info->units.push_back(u);
    }
    if (parts > 1) {
      slot += parts;
      ++counter;
    }
  }
  // heaviest units first so that the long runs start early
  std::stable_sort(info->units.begin(), info->units.end(),
                   [](const AttnUnit& a, const AttnUnit& b) { return a.weight > b.weight; });
  // Between one and two units per CU: the first 256 workgroups take a CU
  // each, and workgroup 256 + j shares the CU of workgroup j (same XCD, the
  // dispatch's second pass).  A unit that shares its CU runs its key blocks
  // slower (kPairCost, against 1 alone) until its partner ends.  The lightest
  // units are already last; moving the lightest of the first pass to the
  // front gives them, rather than the heaviest, a partner.  The order with the
  // shorter estimated longest CU is kept.
  const int64_t n_units = (int64_t)info->units.size(), first = kCUs / 2;
  if (n_units > first && n_units <= kCUs) {
    constexpr double kPairCost = 1.5;
    const int64_t m = n_units - first;
    auto longest = [&](const std::vector<AttnUnit>& u) {
      double t = 0;
      for (int64_t j = 0; j < first; ++j) {
        double c = u[(size_t)j].weight;
        if (j < m) {
          const double a = u[(size_t)j].weight, b = u[(size_t)(first + j)].weight;
          c = kPairCost * std::min(a, b) + (std::max(a, b) - std::min(a, b));
        }
        t = std::max(t, c);
      }
      return t;
    };
    std::vector<AttnUnit> rot = info->units;
    std::rotate(rot.begin(), rot.begin() + (first - m), rot.begin() + first);
    if (longest(rot) < longest(info->units)) info->units.swap(rot);
  }
  info->slots = slot;
  info->counters = counter;
  return EA_OK;
}

// Look up or create the plan of a join-agg call.
// Look up the plan of a join-agg configuration.  With build set, a missing
// plan is created: its tables are uploaded, the GPU join enumerator runs on
// stream s and the host waits for it (and, for attention, sizes the work
// units from the GPU's group offsets).  Without build, a missing plan is
// EA_ERR_NOPLAN: the enqueue path never allocates or synchronizes.
int get_joinagg_plan(const char* spec_str, const Spec& sp, int32_t join_op, int32_t agg_op,
                     const ea_relation* const* ops, const ea_params* prm, const OpInfo& oi, bool build,
                     hipStream_t s, Plan** out) {
  int dev = 0;
  EA_HIP_TRY(hipGetDevice(&dev));
  std::ostringstream k;
  k << "J|" << dev << "|" << spec_str << "|" << join_op << "|" << agg_op << "|" << oi.causal << oi.join_causal
    << "|g" << oi.gqa << "|s";
  for (int64_t e : oi.seq_ends) k << e << ",";
  for (int o = 0; o <= sp.n_in; ++o) key_rel(k, ops[o]);
  const ea_relation* res = prm ? prm->residual : nullptr;
  if (res && (oi.kind == K_GEMM || oi.kind == K_GENERIC)) k << "|res" << res->dtype;
  const std::string key = k.str();
  std::lock_guard<std::mutex> lk(g_cache_mu);
  auto it = cache().find(key);
  if (it != cache().end()) {
    *out = it->second.get();
    return EA_OK;
  }
  if (!build)
    return fail(EA_ERR_NOPLAN, "join-agg '%s' is not planned on device %d: call ea_joinagg_workspace first", spec_str,
                dev);
  JoinInfo ji;
  int e = analyze_join(sp, ops, oi.group, &ji);
  if (e) return e;
  Image img;
  JoinSections js;
  auto p = std::make_unique<Plan>();
  p->kind = oi.kind;
  p->n_in = sp.n_in;
  p->b_kmajor = oi.b_kmajor;
  e = build_join(sp, ops, ji, oi, &img, &js, &p->n_groups, &p->tuple_cap);
  if (e) return e;
  Extra ex;
  switch (oi.kind) {
    case K_GENERIC: e = build_generic(sp, join_op, agg_op, ops, ji, res, &img, &ex); break;
    case K_GEMM: {
      const bool swiglu = join_op == EA_OP_SWIGLU;
      int tn = swiglu ? kGemmTNSwiglu : kGemmTN;
      // direct-to-LDS kernel: contracted block extents multiples of 32, at
      // most kGemmMaxTuples tuples per group (staged in LDS) and operand
      // blocks below 4 GiB (32-bit lane offsets); else the register-staged one
      bool k32 = true;
      for (int64_t v : ops[0]->splits[1]) k32 &= v % 32 == 0;
      bool small = true;
      for (int i = 0; i < sp.n_in; ++i) small &= max_block_bytes(ops[i]) < (int64_t(1) << 32);
      p->gemm_direct = k32 && ops[0]->nb[1] <= kGemmMaxTuples && small;
      GemmPlanInfo gi = gemm_units(ops[0], ops[sp.n_in], tn);
      GemmDlPlan dl;
      if (p->gemm_direct) dl = gemm_units_dl(ops[0], ops[sp.n_in], tn, gi);
      if (p->gemm_direct && !swiglu) {
        // 256 x 128 tiles: twice the workgroups for the same work, so fewer
        // split sums (or none) where 256-wide tiles leave CUs idle; a K step
        // of one costs kNarrowStep of a 256-wide one (the operand bytes per
        // MFMA rise by half)
        const GemmPlanInfo gn = gemm_units(ops[0], ops[sp.n_in], kGemmTNSwiglu, kNarrowStep);
        const GemmDlPlan dn = gemm_units_dl(ops[0], ops[sp.n_in], kGemmTNSwiglu, gn, kNarrowStep);
        const char* force = getenv("EA_GEMM_TILE_N");  // 128 or 256 overrides the model when a plan is built
        const bool narrow = force ? atoi(force) == 128 : dn.cost < dl.cost;
        if (narrow) {
          tn = kGemmTNSwiglu;
          gi = gn;
          dl = dn;
        }
      }
      p->gemm_tn = tn;
      p->gemm_parts = gi.parts;
      int64_t slots = gi.slots;
      if (p->gemm_direct) {
        ex.work = img.put_vec(dl.units);
        ex.n_work = (int64_t)dl.units.size();
        ex.meta = img.put_zero((size_t)p->tuple_cap * sizeof(GemmTupleMeta));
        slots = dl.slots;
        p->ws_counters = dl.counters;
      } else {
        ex.work = img.put_vec(gi.units);
        ex.n_work = (int64_t)gi.units.size();
        p->ws_counters = gi.counters;
      }
      // fp32 partial tiles of split keys in the workspace
      p->ws_partial_bytes = slots * kGemmTM * kGemmTN * (int64_t)sizeof(float);
      break;
    }
    case K_GEMM32: {  // square tiles of every output block
      std::vector<Gemm32Work> work;
      const ea_relation* c = ops[sp.n_in];
      int32_t co[kMaxRank];
      for (int64_t b = 0; b < c->nblocks; ++b) {
        block_coords(c, b, co);
        const int64_t me = c->splits[0][co[0] + 1] - c->splits[0][co[0]];
        const int64_t ne = c->splits[1][co[1] + 1] - c->splits[1][co[1]];
        for (int64_t m0 = 0; m0 < me; m0 += kGemm32Tile)
          for (int64_t n0 = 0; n0 < ne; n0 += kGemm32Tile)
            work.push_back(Gemm32Work{(int32_t)b, (int32_t)m0, (int32_t)n0, 0});
      }
      ex.work = img.put_vec(work);
      ex.n_work = (int64_t)work.size();
      break;
    }
    case K_RMSNORM:
    case K_SOFTMAX: e = build_rows(sp, ops, oi, &img, &ex, &p->rows); break;
    case K_ATTENTION: break;  // work units follow the GPU join (below)
    default: e = fail(EA_ERR_UNSUPPORTED, "internal: unknown plan kind");
  }
  if (e) return e;
  e = plan_upload(p.get(), img, s);
  if (e) return e;
  p->d_desc = ex.desc ? p->dmem + ex.desc : nullptr;
  p->d_work = p->dmem + ex.work;
  p->n_work = ex.n_work;
  e = finish_join(p.get(), js, sp.n_in + 1, s);
  if (e) return e;
  if (oi.kind == K_GEMM && p->gemm_direct) {
    // resolve the join into the work list: per-tuple operand blocks and
    // each segment's place in its group's walk (the join has completed)
    p->d_gemm_meta = (GemmTupleMeta*)(p->dmem + ex.meta);
    GemmArgs a;
    memset(&a, 0, sizeof(a));
    a.tuples = p->d_tuples;
    a.goff = p->d_goff;
    a.count = p->d_count;
    a.blk_a = p->d_blk[0];
    a.blk_b = p->d_blk[1];
    a.swiglu = join_op == EA_OP_SWIGLU;
    if (a.swiglu) a.blk_b2 = p->d_blk[2];
    a.tuple_stride = sp.n_in + 1;
    a.n_units = (int32_t)p->n_work;
    a.meta = p->d_gemm_meta;
    EA_HIP_TRY(launch_gemm_prep(a, (GemmUnit*)(p->dmem + ex.work), p->tuple_cap, s));
    EA_HIP_TRY(hipStreamSynchronize(s));
  }
  if (oi.kind == K_ATTENTION) {
    // units from the GPU-built group offsets (the join has completed)
    std::vector<int32_t> goff((size_t)p->n_groups + 1);
    EA_HIP_TRY(hipMemcpyAsync(goff.data(), p->d_goff, goff.size() * sizeof(int32_t), hipMemcpyDeviceToHost, s));
    EA_HIP_TRY(hipStreamSynchronize(s));
    AttnPlanInfo ai;
    e = attention_units(ops[0], goff, &ai);
    if (e) return e;
    Image img2;
    const size_t uoff = img2.put_vec(ai.units);
    const size_t moff = img2.put_zero(ai.units.size() * sizeof(AttnUnitMeta));
    const size_t foff = img2.put_zero(sizeof(int32_t));
    e = upload_image(img2, &p->dmem2, s);
    if (e) return e;
    p->d_work = p->dmem2 + uoff;
    p->n_work = (int64_t)ai.units.size();
    p->attn_meta = (AttnUnitMeta*)(p->dmem2 + moff);
    const int64_t slots = ai.slots;
    p->ws_counters = ai.counters;
    p->ws_part_ml = (size_t)slots * 128 * 128 * sizeof(float);
    p->ws_partial_bytes = slots ? (int64_t)p->ws_part_ml + slots * 128 * 2 * (int64_t)sizeof(float) : 0;
    AttnArgs a;
    memset(&a, 0, sizeof(a));
    a.tuples = p->d_tuples;
    a.goff = p->d_goff;
    a.blk_q = p->d_blk[0];
    a.blk_k = p->d_blk[1];
    a.blk_v = p->d_blk[2];
    a.blk_o = p->d_blk[3];
    a.units = (const AttnUnit*)p->d_work;
    a.n_units = (int32_t)p->n_work;
    a.q_dim = oi.q_dim;
    a.k_dim = oi.k_dim;
    a.causal = oi.causal;  // the walk's causal cut and its unmasked leading chunks (a plan holds one rule)
    a.meta = p->attn_meta;
    a.overflow = (int32_t*)(p->dmem2 + foff);
    EA_HIP_TRY(launch_attention_prep(a, s));
    int32_t overflow = 0;
    EA_HIP_TRY(hipMemcpyAsync(&overflow, a.overflow, sizeof(int32_t), hipMemcpyDeviceToHost, s));
    EA_HIP_TRY(hipStreamSynchronize(s));
    if (overflow)
      return fail(EA_ERR_HIP, "internal: an attention unit holds more than %d key blocks", kAttnMaxUnitTuples);
  }
  if (p->ws_counters * (int64_t)sizeof(int32_t) > kWsCounterBytes)
    return fail(EA_ERR_UNSUPPORTED, "plan needs %lld split-key counters, above the workspace's %lld",
                (long long)p->ws_counters, (long long)(kWsCounterBytes / (int64_t)sizeof(int32_t)));
  *out = p.get();
  cache()[key] = std::move(p);
  return EA_OK;
}

int check_rel(const ea_relation* r, const char* what, bool need_data) {
  if (!r) return fail(EA_ERR_ARG, "NULL %s relation", what);
  if (need_data && !r->data) return fail(EA_ERR_ARG, "%s relation has no data", what);
  return EA_OK;
}

// Common front half of ea_joinagg / ea_join_tuples: validation + plan.
int prepare(const char* spec, int32_t join_op, int32_t agg_op, int32_t n_in, const ea_relation* const* in,
            const ea_relation* out, const ea_params* prm, bool need_data, bool build, hipStream_t s, Spec* sp,
            OpInfo* oi, Plan** plan) {
  if (!spec) return fail(EA_ERR_ARG, "NULL spec");
  if (n_in < 1 || n_in > kMaxIn || !in) return fail(EA_ERR_ARG, "n_in %d outside [1, %d] or NULL inputs", n_in, kMaxIn);
  for (int i = 0; i < n_in; ++i) {
    int e = check_rel(in[i], "input", need_data);
    if (e) return e;
  }
  int e = check_rel(out, "output", need_data);
  if (e) return e;
  e = parse_spec(spec, sp);
  if (e) return e;
  if (sp->n_in != n_in) return fail(EA_ERR_SPEC, "spec '%s' has %d inputs, call passes %d", spec, sp->n_in, n_in);
  const ea_relation* ops[kMaxOps];
  for (int i = 0; i < n_in; ++i) ops[i] = in[i];
  ops[n_in] = out;
  for (int o = 0; o <= n_in; ++o)
    if (ops[o]->rank != sp->rank[o])
      return fail(EA_ERR_SPEC, "operand %d has rank %d but the spec gives it %d letters", o, ops[o]->rank,
                  sp->rank[o]);
  if (prm && prm->store != EA_STORE_CACHED && prm->store != EA_STORE_STREAM)
    return fail(EA_ERR_ARG, "params.store must be EA_STORE_CACHED or EA_STORE_STREAM");
  if (prm && prm->gqa_group < 0) return fail(EA_ERR_ARG, "params.gqa_group %d is negative", prm->gqa_group);
  if (prm && join_op != EA_OP_ATTENTION && (prm->gqa_group > 1 || prm->n_seq != 0))
    return fail(EA_ERR_ARG, "params.gqa_group and params.n_seq apply to EA_OP_ATTENTION only");
  e = classify(*sp, join_op, agg_op, ops, prm, oi);
  if (e) return e;
  // join validation runs here too, before any HIP call
  JoinInfo ji;
  e = analyze_join(*sp, ops, oi->group, &ji);
  if (e) return e;
  if (!plan) return EA_OK;
  return get_joinagg_plan(spec, *sp, join_op, agg_op, ops, prm, *oi, build, s, plan);
}

// Validate a run of a planned join-agg and find its plan (never building it).
int lookup_run(const char* spec, int32_t join_op, int32_t agg_op, int32_t n_in, const ea_relation* const* in,
               const ea_relation* out, const ea_params* params, hipStream_t s, OpInfo* oi, Plan** plan) {
  Spec sp;
  return prepare(spec, join_op, agg_op, n_in, in, out, params, true, false, s, &sp, oi, plan);
}

// ---------------------------------------------------------------------------
// Split-key workspace of ea_joinagg_noalloc: a fixed device array in the
// library's code object, so that the entry point allocates nothing.  Each
// device holds its own copy at its own address, found once per device with
// hipGetSymbolAddress; host code uses that address only, never the array's
// name (a host-side stand-in).
// ---------------------------------------------------------------------------
constexpr int64_t kNoAllocScratchBytes = EA_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

__global__ void zero_words_kernel(int32_t* p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

std::mutex g_scratch_mu;
std::map<int, char*>& scratch_addr() {
  static auto* m = new std::map<int, char*>();  // device -> its copy's address; intentionally leaked at exit
  return *m;
}

// Address of the current device's copy of the array (looked up on the
// device's first call, with that device current).
int noalloc_scratch(char** out) {
  int dev = 0;
  EA_HIP_TRY(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  auto it = scratch_addr().find(dev);
  if (it == scratch_addr().end()) {
    void* p = nullptr;
    EA_HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p || (uintptr_t)p % 256) return fail(EA_ERR_HIP, "scratch array of device %d at %p", dev, p);
    it = scratch_addr().emplace(dev, (char*)p).first;
  }
  *out = it->second;
  return EA_OK;
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

int ea_version(void) { return EA_VERSION; }

const char* ea_last_error(void) { return g_err.c_str(); }

int ea_dtype_size(int32_t dtype) {
  int s = dtype_size(dtype);
  if (s < 0) return fail(EA_ERR_DTYPE, "unknown dtype %d", dtype);
  return s;
}

int ea_layout_nbytes(int32_t rank, const int64_t* shape, int32_t dtype, const int32_t* nblocks,
                     const int64_t* splits, int64_t* nbytes) {
  if (!nbytes) return fail(EA_ERR_ARG, "NULL nbytes");
  if (dtype_size(dtype) < 0) return fail(EA_ERR_DTYPE, "unknown dtype %d", dtype);
  int e = check_partition(rank, shape, nblocks, splits);
  if (e) return e;
  ea_relation r;
  r.rank = rank;
  r.dtype = dtype;
  const int64_t* s = splits;
  for (int d = 0; d < rank; ++d) {
    r.nb[d] = nblocks[d];
    r.splits[d].assign(s, s + nblocks[d] + 1);
    s += nblocks[d] + 1;
  }
  fill_layout(&r);
  *nbytes = r.nbytes;
  return ok();
}

int ea_relation_create(int32_t rank, const int64_t* shape, int32_t dtype, const int32_t* nblocks,
                       const int64_t* splits, void* data, int64_t capacity, ea_relation** out) {
  if (!out) return fail(EA_ERR_ARG, "NULL out handle");
  *out = nullptr;
  if (dtype_size(dtype) < 0) return fail(EA_ERR_DTYPE, "unknown dtype %d", dtype);
  int e = check_partition(rank, shape, nblocks, splits);
  if (e) return e;
  auto r = std::make_unique<ea_relation>();
  r->rank = rank;
  r->dtype = dtype;
  const int64_t* s = splits;
  for (int d = 0; d < rank; ++d) {
    r->shape[d] = shape[d];
    r->nb[d] = nblocks[d];
    r->splits[d].assign(s, s + nblocks[d] + 1);
    s += nblocks[d] + 1;
  }
  fill_layout(r.get());
  if (data) {
    if ((uintptr_t)data % 256) return fail(EA_ERR_ARG, "relation data must be 256-byte aligned");
    if (capacity < r->nbytes)
      return fail(EA_ERR_CAPACITY, "capacity %lld below the layout's %lld bytes", (long long)capacity,
                  (long long)r->nbytes);
  }
  r->data = data;
  r->capacity = capacity;
  *out = r.release();
  return ok();
}

int ea_relation_destroy(ea_relation* rel) {
  delete rel;
  return ok();
}

int ea_relation_set_data(ea_relation* rel, void* data, int64_t capacity) {
  if (!rel) return fail(EA_ERR_ARG, "NULL relation");
  if (data && (uintptr_t)data % 256) return fail(EA_ERR_ARG, "relation data must be 256-byte aligned");
  if (data && capacity < rel->nbytes)
    return fail(EA_ERR_CAPACITY, "capacity %lld below the layout's %lld bytes", (long long)capacity,
                (long long)rel->nbytes);
  rel->data = data;
  rel->capacity = capacity;
  return ok();
}

int ea_relation_num_blocks(const ea_relation* rel, int64_t* n) {
  if (!rel || !n) return fail(EA_ERR_ARG, "NULL argument");
  *n = rel->nblocks;
  return ok();
}

int ea_relation_nbytes(const ea_relation* rel, int64_t* nbytes) {
  if (!rel || !nbytes) return fail(EA_ERR_ARG, "NULL argument");
  *nbytes = rel->nbytes;
  return ok();
}

int ea_relation_block(const ea_relation* rel, int64_t b, int64_t* lo, int64_t* hi, int64_t* byte_off) {
  if (!rel) return fail(EA_ERR_ARG, "NULL relation");
  if (b < 0 || b >= rel->nblocks) return fail(EA_ERR_ARG, "block %lld outside [0, %lld)", (long long)b,
                                              (long long)rel->nblocks);
  int32_t c[kMaxRank];
  block_coords(rel, b, c);
  for (int d = 0; d < rel->rank; ++d) {
    if (lo) lo[d] = rel->splits[d][c[d]];
    if (hi) hi[d] = rel->splits[d][c[d] + 1];
  }
  if (byte_off) *byte_off = rel->off[(size_t)b];
  return ok();
}

int ea_overlay(int32_t rank, const int32_t* nblocks_a, const int64_t* splits_a, const int32_t* nblocks_b,
               const int64_t* splits_b, int32_t* nblocks_out, int64_t* splits_out) {
  if (rank < 1 || rank > kMaxRank || !nblocks_a || !splits_a || !nblocks_b || !splits_b || !nblocks_out ||
      !splits_out)
    return fail(EA_ERR_ARG, "bad overlay arguments");
  const int64_t* sa = splits_a;
  const int64_t* sb = splits_b;
  int64_t* so = splits_out;
  for (int d = 0; d < rank; ++d) {
    if (nblocks_a[d] < 1 || nblocks_b[d] < 1) return fail(EA_ERR_PARTITION, "dim %d has no blocks", d);
    if (sa[nblocks_a[d]] != sb[nblocks_b[d]]) return fail(EA_ERR_ARG, "dim %d: extents differ", d);
    std::vector<int64_t> u(sa, sa + nblocks_a[d] + 1);
    u.insert(u.end(), sb, sb + nblocks_b[d] + 1);
    std::sort(u.begin(), u.end());
    u.erase(std::unique(u.begin(), u.end()), u.end());
    nblocks_out[d] = (int32_t)u.size() - 1;
    std::copy(u.begin(), u.end(), so);
    so += u.size();
    sa += nblocks_a[d] + 1;
    sb += nblocks_b[d] + 1;
  }
  return ok();
}

int ea_join_tuples(const char* spec, int32_t join_op, int32_t n_in, const ea_relation* const* in,
                   const ea_relation* out, const ea_params* params, int32_t* tuples, int64_t cap,
                   int64_t* group_off, int64_t gcap, int64_t* n_tuples, int64_t* n_groups, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  int32_t agg = EA_AGG_SUM;
  if (join_op == EA_OP_SOFTMAX || join_op == EA_OP_ATTENTION) agg = EA_AGG_LSE;
  if ((join_op == EA_JOIN_MUL || join_op == EA_JOIN_ADD) && spec) {
    // NONE when nothing is contracted, so that pure joins can be inspected too
    Spec sp;
    if (parse_spec(spec, &sp) == EA_OK) {
      bool contracted = false;
      for (int i = 0; i < sp.n_in; ++i)
        for (int d = 0; d < sp.rank[i]; ++d) contracted |= find_dim(sp, sp.n_in, sp.let[i][d]) < 0;
      if (!contracted) agg = EA_AGG_NONE;
    }
  }
  Spec sp;
  OpInfo oi;
  Plan* plan = nullptr;
  int e = prepare(spec, join_op, agg, n_in, in, out, params, false, true, s, &sp, &oi, &plan);
  if (e) return e;
  int32_t count = 0;
  EA_HIP_TRY(hipMemcpyAsync(&count, plan->d_count, sizeof(int32_t), hipMemcpyDeviceToHost, s));
  EA_HIP_TRY(hipStreamSynchronize(s));
  if (n_tuples) *n_tuples = count;
  if (n_groups) *n_groups = plan->n_groups;
  if (!tuples || !group_off) return fail(EA_ERR_ARG, "NULL tuple or group buffer");
  if (cap < count || gcap < plan->n_groups + 1)
    return fail(EA_ERR_CAPACITY, "need %d tuples and %lld group offsets", count, (long long)plan->n_groups + 1);
  const int stride = plan->n_in + 1;
  EA_HIP_TRY(hipMemcpyAsync(tuples, plan->d_tuples, (size_t)count * stride * sizeof(int32_t),
                            hipMemcpyDeviceToDevice, s));
  // widen the int32 offsets to int64 through the host (test path only)
  std::vector<int32_t> g32((size_t)plan->n_groups + 1);
  EA_HIP_TRY(hipMemcpyAsync(g32.data(), plan->d_goff, g32.size() * sizeof(int32_t), hipMemcpyDeviceToHost, s));
  EA_HIP_TRY(hipStreamSynchronize(s));
  std::vector<int64_t> g64(g32.begin(), g32.end());
  EA_HIP_TRY(hipMemcpyAsync(group_off, g64.data(), g64.size() * sizeof(int64_t), hipMemcpyHostToDevice, s));
  EA_HIP_TRY(hipStreamSynchronize(s));
  return ok();
}

}  // extern "C"

namespace {

// Enqueue the kernels of a planned join-agg on stream s.  ws: the split-key
// workspace (counters at its start, partial results from kWsCounterBytes),
// at least plan->ws_bytes() bytes, or null when the plan needs none.
int run_planned(const Plan* plan, int32_t join_op, int32_t n_in, const ea_relation* const* in, ea_relation* out,
                const ea_params* params, const OpInfo& oi, char* ws, hipStream_t s) {
  const ea_relation* res = params ? params->residual : nullptr;
  switch (plan->kind) {
    case K_GENERIC: {
      GenArgs a;
      memset(&a, 0, sizeof(a));
      a.desc = (const GenDesc*)plan->d_desc;
      a.tuples = plan->d_tuples;
      a.goff = plan->d_goff;
      for (int o = 0; o <= n_in; ++o) a.blk[o] = plan->d_blk[o];
      for (int i = 0; i < n_in; ++i) a.in[i] = (const char*)in[i]->data;
      a.out = (char*)out->data;
      a.res = res ? (const char*)res->data : nullptr;
      a.work = (const GenWork*)plan->d_work;
      a.n_work = plan->n_work;
      EA_HIP_TRY(launch_generic(a, s));
      break;
    }
    case K_GEMM: {
      GemmArgs a;
      memset(&a, 0, sizeof(a));
      a.tuples = plan->d_tuples;
      a.goff = plan->d_goff;
      a.blk_a = plan->d_blk[0];
      a.blk_b = plan->d_blk[1];
      a.a = (const char*)in[0]->data;
      a.b = (const char*)in[1]->data;
      a.swiglu = join_op == EA_OP_SWIGLU;
      if (a.swiglu) {
        a.blk_b2 = plan->d_blk[2];
        a.b2 = (const char*)in[2]->data;
      }
      a.blk_c = plan->d_blk[n_in];
      a.c = (char*)out->data;
      a.res = res ? (const char*)res->data : nullptr;
      a.dt_res = res ? res->dtype : 0;
      a.direct = plan->gemm_direct;
      a.tile_n = plan->gemm_tn;
      a.meta = plan->d_gemm_meta;
      if (a.direct) {
        a.units = (const GemmUnit*)plan->d_work;
        a.n_units = (int32_t)plan->n_work;
      } else {
        a.tiles = (const GemmTile*)plan->d_work;
        a.n_tiles = (int32_t)plan->n_work;
      }
      a.tuple_stride = n_in + 1;
      a.b_kmajor = plan->b_kmajor;
      a.dt_in = in[0]->dtype;
      a.dt_out = out->dtype;
      a.partials = (float*)(ws + kWsCounterBytes);
      a.counters = (int32_t*)ws;
      EA_HIP_TRY(launch_gemm(a, s));
      break;
    }
    case K_GEMM32: {
      Gemm32Args a;
      memset(&a, 0, sizeof(a));
      a.tuples = plan->d_tuples;
      a.goff = plan->d_goff;
      a.blk_a = plan->d_blk[0];
      a.blk_b = plan->d_blk[1];
      a.blk_c = plan->d_blk[2];
      a.a = (const char*)in[0]->data;
      a.b = (const char*)in[1]->data;
      a.c = (char*)out->data;
      a.work = (const Gemm32Work*)plan->d_work;
      a.n_work = plan->n_work;
      a.tuple_stride = 3;
      a.b_kmajor = plan->b_kmajor;
      a.dt_out = out->dtype;
      EA_HIP_TRY(launch_gemm32(a, s));
      break;
    }
    case K_RMSNORM:
    case K_SOFTMAX: {
      RowArgs a;
      memset(&a, 0, sizeof(a));
      a.tuples = plan->d_tuples;
      a.goff = plan->d_goff;
      a.blk_x = plan->d_blk[0];
      a.x = (const char*)in[0]->data;
      a.dt_x = in[0]->dtype;
      if (plan->kind == K_RMSNORM) {
        a.blk_w = plan->d_blk[1];
        a.w = (const char*)in[1]->data;
        a.dt_w = in[1]->dtype;
        a.eps = params->eps;
      }
      a.blk_y = plan->d_blk[n_in];
      a.y = (char*)out->data;
      a.dt_y = out->dtype;
      a.tasks = (const RowTask*)plan->d_work;
      a.n_rowtasks = (int32_t)plan->n_work;
      a.tuple_stride = n_in + 1;
      a.rank = out->rank;
      a.causal = oi.causal;
      a.row_len = plan->rows.row_len;
      a.vec = plan->rows.vec;
      a.seg_chunks = plan->rows.cps;
      a.seg_inv = a.seg_chunks > 0 ? 1.0f / (float)a.seg_chunks : 0.0f;
      a.affine = plan->rows.affine;
      a.stream_out = params ? params->store : 0;
      a.seg_len = plan->rows.seg_len;
      a.nseg = plan->rows.nseg;
      a.xs = plan->rows.xs;
      a.ys = plan->rows.ys;
      a.ws = plan->rows.ws;
      a.wbase = plan->rows.wbase;
      EA_HIP_TRY(plan->kind == K_RMSNORM ? launch_rmsnorm(a, s) : launch_softmax(a, s));
      break;
    }
    case K_ATTENTION: {
      AttnArgs a;
      memset(&a, 0, sizeof(a));
      a.tuples = plan->d_tuples;
      a.goff = plan->d_goff;
      a.blk_q = plan->d_blk[0];
      a.blk_k = plan->d_blk[1];
      a.blk_v = plan->d_blk[2];
      a.blk_o = plan->d_blk[3];
      a.q = (const char*)in[0]->data;
      a.k = (const char*)in[1]->data;
      a.v = (const char*)in[2]->data;
      a.o = (char*)out->data;
      a.units = (const AttnUnit*)plan->d_work;
      a.n_units = (int32_t)plan->n_work;
      a.causal = oi.causal;
      a.q_dim = oi.q_dim;
      a.k_dim = oi.k_dim;
      a.scale = params->scale;
      a.part_o = (float*)(ws + kWsCounterBytes);
      a.part_ml = (float*)(ws + kWsCounterBytes + plan->ws_part_ml);
      a.counters = (int32_t*)ws;
      a.dt_o = out->dtype;
      a.meta = plan->attn_meta;
      EA_HIP_TRY(launch_attention(a, s));
      break;
    }
    default:
      return fail(EA_ERR_UNSUPPORTED, "internal: plan kind %d", (int)plan->kind);
  }
  return EA_OK;
}

}  // namespace

extern "C" {


int ea_joinagg_workspace(const char* spec, int32_t join_op, int32_t agg_op, int32_t n_in,
                         const ea_relation* const* in, const ea_relation* out, const ea_params* params,
                         int64_t* ws_bytes, void* stream) {
  if (!ws_bytes) return fail(EA_ERR_ARG, "NULL ws_bytes");
  *ws_bytes = 0;
  Spec sp;
  OpInfo oi;
  Plan* plan = nullptr;
  int e = prepare(spec, join_op, agg_op, n_in, in, out, params, false, true, (hipStream_t)stream, &sp, &oi, &plan);
  if (e) return e;
  *ws_bytes = plan->ws_bytes();
  return ok();
}

int ea_joinagg(const char* spec, int32_t join_op, int32_t agg_op, int32_t n_in, const ea_relation* const* in,
               ea_relation* out, const ea_params* params, void* workspace, int64_t ws_bytes, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  OpInfo oi;
  Plan* plan = nullptr;
  int e = lookup_run(spec, join_op, agg_op, n_in, in, out, params, s, &oi, &plan);
  if (e) return e;
  const int64_t need = plan->ws_bytes();
  if (need) {
    if (!workspace) return fail(EA_ERR_ARG, "this join-agg needs a workspace of %lld bytes", (long long)need);
    if ((uintptr_t)workspace % 256) return fail(EA_ERR_ARG, "workspace must be 256-byte aligned");
    if (ws_bytes < need)
      return fail(EA_ERR_CAPACITY, "workspace of %lld bytes below the %lld this join-agg needs", (long long)ws_bytes,
                  (long long)need);
  }
  e = run_planned(plan, join_op, n_in, in, out, params, oi, need ? (char*)workspace : nullptr, s);
  if (e) return e;
  return ok();
}

int ea_joinagg_noalloc(const char* spec, int32_t join_op, int32_t agg_op, int32_t n_in, const ea_relation* const* in,
                       ea_relation* out, const ea_params* params, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  OpInfo oi;
  Plan* plan = nullptr;
  int e = lookup_run(spec, join_op, agg_op, n_in, in, out, params, s, &oi, &plan);
  if (e) return e;
  const int64_t need = plan->ws_bytes();
  char* ws = nullptr;
  if (need) {
    if (need > kNoAllocScratchBytes)
      return fail(EA_ERR_CAPACITY, "this join-agg needs %lld bytes of workspace, above the %lld of ea_joinagg_noalloc",
                  (long long)need, (long long)kNoAllocScratchBytes);
    e = noalloc_scratch(&ws);
    if (e) return e;
    // the counters start at zero whatever an earlier call left (a fill
    // kernel, not a memset node, so that the call can be captured)
    if (plan->ws_counters) {
      const int64_t n = plan->ws_counters;
      hipLaunchKernelGGL(zero_words_kernel, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0, s, (int32_t*)ws, n);
      EA_HIP_TRY(hipGetLastError());
    }
  }
  e = run_planned(plan, join_op, n_in, in, out, params, oi, ws, s);
  if (e) return e;
  return ok();
}

int ea_repartition(const ea_relation* src, ea_relation* dst, void* stream) {
  return ea_repartition_ex(src, dst, EA_STORE_CACHED, stream);
}

}  // extern "C"

namespace {

int check_repartition(const ea_relation* src, const ea_relation* dst, bool need_data) {
  if (!src || !dst) return fail(EA_ERR_ARG, "NULL relation");
  if (need_data && (!src->data || !dst->data)) return fail(EA_ERR_ARG, "relation has no data");
  if (src->rank != dst->rank || src->dtype != dst->dtype)
    return fail(EA_ERR_ARG, "source and destination differ in rank or dtype");
  for (int d = 0; d < src->rank; ++d)
    if (src->shape[d] != dst->shape[d]) return fail(EA_ERR_ARG, "source and destination differ in shape");
  if (need_data) {
    const char* a0 = (const char*)src->data;
    const char* b0 = (const char*)dst->data;
    if (a0 < b0 + dst->nbytes && b0 < a0 + src->nbytes)
      return fail(EA_ERR_ARG, "source and destination memory overlap");
  }
  return EA_OK;
}

// The plan of a repartition (its overlay boxes), built when `build` is set.
int get_repartition_plan(const ea_relation* src, const ea_relation* dst, bool build, hipStream_t s, Plan** out) {
  int dev = 0;
  EA_HIP_TRY(hipGetDevice(&dev));
  std::ostringstream k;
  k << "R|" << dev;
  key_rel(k, src);
  key_rel(k, dst);
  const std::string key = k.str();
  Plan* plan = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_cache_mu);
    auto it = cache().find(key);
    if (it != cache().end()) plan = it->second.get();
    if (!plan && !build)
      return fail(EA_ERR_NOPLAN, "repartition is not planned on device %d: call ea_repartition_plan first", dev);
    if (!plan) {
      // Overlay (Section 5.3): cut every dim at the union of both partitions'
      // split points.  A box = the intersection of one source block and one
      // destination block = a union of overlay atoms; it is copied row by row.
      const int R = src->rank;
      const int es = dtype_size(src->dtype);
      std::vector<RepTask> tasks;
      int64_t rel_bytes = es;
      for (int d = 0; d < R; ++d) rel_bytes *= src->shape[d];
      const bool small_tasks = rel_bytes < kRepLargeBytes;
      int32_t cd[kMaxRank];
      std::vector<DevBlk> sb = dev_blocks(src);
      for (int64_t b = 0; b < dst->nblocks; ++b) {
        block_coords(dst, b, cd);
        // source blocks overlapping destination block b: per dim, the source
        // intervals that meet [dlo, dhi)
        std::vector<int32_t> lo_i(R), hi_i(R);
        for (int d = 0; d < R; ++d) {
          const int64_t dlo = dst->splits[d][cd[d]], dhi = dst->splits[d][cd[d] + 1];
          const auto& ss = src->splits[d];
          int first = (int)(std::upper_bound(ss.begin(), ss.end(), dlo) - ss.begin()) - 1;
          int last = (int)(std::lower_bound(ss.begin(), ss.end(), dhi) - ss.begin()) - 1;
          lo_i[d] = first;
          hi_i[d] = last + 1;
        }
        std::vector<int32_t> cs(lo_i);
        while (true) {
          int64_t sbi = 0;
          for (int d = 0; d < R; ++d) sbi = sbi * src->nb[d] + cs[d];
          const DevBlk& S = sb[(size_t)sbi];
          int64_t blo[kMaxRank], bext[kMaxRank];
          for (int d = 0; d < R; ++d) {
            const int64_t dlo = dst->splits[d][cd[d]], dhi = dst->splits[d][cd[d] + 1];
            const int64_t slo = S.lo[d], shi = S.lo[d] + S.ext[d];
            blo[d] = std::max(dlo, slo);
            bext[d] = std::min(dhi, shi) - blo[d];
          }
          // row-major strides (elements) inside each block
          int64_t sst[kMaxRank], dst_st[kMaxRank];
          sst[R - 1] = dst_st[R - 1] = 1;
          for (int d = R - 2; d >= 0; --d) {
            sst[d] = sst[d + 1] * S.ext[d + 1];
            dst_st[d] = dst_st[d + 1] * (dst->splits[d + 1][cd[d + 1] + 1] - dst->splits[d + 1][cd[d + 1]]);
          }
          RepTask t;
          memset(&t, 0, sizeof(t));
          int64_t so = 0, dofs = 0;
          for (int d = 0; d < R; ++d) {
            so += (blo[d] - S.lo[d]) * sst[d];
            dofs += (blo[d] - dst->splits[d][cd[d]]) * dst_st[d];
          }
          t.src_off = S.off + so * es;
          t.dst_off = dst->off[(size_t)b] + dofs * es;
          // merge trailing dims that are contiguous in both blocks into the row
          int last = R - 1;
          int64_t row_elems = bext[R - 1];
          while (last > 0 && bext[last] == S.ext[last] &&
                 bext[last] == dst->splits[last][cd[last] + 1] - dst->splits[last][cd[last]]) {
            row_elems *= bext[last - 1];
            --last;
          }
          t.n_outer = last;
          int64_t rows = 1;
          for (int d = 0; d < last; ++d) {
            t.outer_ext[d] = (int32_t)bext[d];
            t.src_stride[d] = sst[d] * es;
            t.dst_stride[d] = dst_st[d] * es;
            rows *= bext[d];
          }
          const int64_t rb = row_elems * es;
          if (rb > INT32_MAX || rows > INT32_MAX) return fail(EA_ERR_UNSUPPORTED, "repartition box too large");
          if (rows * rb > INT32_MAX) return fail(EA_ERR_UNSUPPORTED, "repartition box too large");
          t.row_bytes = (int32_t)rb;
          t.row_shift = -1;
          for (int b = 0; b < 31; ++b)
            if (((int64_t)1 << b) == rb) t.row_shift = b;
          int vec = 16;
          auto fits = [&](int64_t v) { return v % vec == 0; };
          while (vec > 1) {
            bool good = fits(t.row_bytes) && fits(t.src_off) && fits(t.dst_off);
            for (int d = 0; d < last; ++d) good = good && fits(t.src_stride[d]) && fits(t.dst_stride[d]);
            if (good) break;
            vec /= 2;
          }
          t.vec = vec;
          // a range of the box per workgroup task (one pass of its 256 lanes)
          const int64_t total = rows * rb, per = small_tasks ? kRepTaskBytesSmall : kRepTaskBytes;
          for (int64_t b0 = 0; b0 < total; b0 += per) {
            RepTask u = t;
            u.begin = (int32_t)b0;
            u.end = (int32_t)std::min(total, b0 + per);
            tasks.push_back(u);
          }
          int d = R - 1;
          while (d >= 0) {
            if (++cs[d] < hi_i[d]) break;
            cs[d] = lo_i[d];
            --d;
          }
          if (d < 0) break;
        }
      }
      Image img;
      const size_t toff = img.put_vec(tasks);
      auto p = std::make_unique<Plan>();
      p->kind = K_REPART;
      p->rep_small = small_tasks;
      int e = plan_upload(p.get(), img, s);
      if (e) return e;
      EA_HIP_TRY(hipStreamSynchronize(s));
      p->d_work = p->dmem + toff;
      p->n_work = (int64_t)tasks.size();
      plan = p.get();
      cache()[key] = std::move(p);
    }
  }
  *out = plan;
  return EA_OK;
}

}  // namespace

extern "C" {

int ea_repartition_plan(const ea_relation* src, const ea_relation* dst, void* stream) {
  int e = check_repartition(src, dst, false);
  if (e) return e;
  Plan* plan = nullptr;
  e = get_repartition_plan(src, dst, true, (hipStream_t)stream, &plan);
  if (e) return e;
  return ok();
}

int ea_repartition_ex(const ea_relation* src, ea_relation* dst, int32_t store, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  if (store != EA_STORE_CACHED && store != EA_STORE_STREAM) return fail(EA_ERR_ARG, "store must be EA_STORE_CACHED or EA_STORE_STREAM");
  int e = check_repartition(src, dst, true);
  if (e) return e;
  Plan* plan = nullptr;
  e = get_repartition_plan(src, dst, false, s, &plan);
  if (e) return e;
  EA_HIP_TRY(launch_repartition((const RepTask*)plan->d_work, plan->n_work, (const char*)src->data,
                                (char*)dst->data, store == EA_STORE_STREAM, plan->rep_small, s));
  return ok();
}

int64_t ea_plan_cache_size(void) {
  std::lock_guard<std::mutex> lk(g_cache_mu);
  return (int64_t)cache().size();
}

int ea_plan_cache_clear(void) {
  std::lock_guard<std::mutex> lk(g_cache_mu);
  cache().clear();
  return ok();
}

}  // extern "C"
