/*
 * ea_oracle.c -- plain CPU oracle for the block join-agg hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
 * baseline leg of the benchmark load this library.  It shares no code, no
 * header and no table with the GPU library: it has its own spec parser, its
 * own block layout code, its own join and its own arithmetic.
 *
 * Every numeric routine computes the dense definition of its result in fp64
 * scalar loops (OpenMP over output rows, no BLAS, no blocking beyond what the
 * definition states).  Blocks matter only where they *are* the result: the
 * block layout, the join's tuple table and the repartition.
 *
 * Paper: "Every Kernel Is a Join: Automatic Multi-GPU Parallelism for AI
 * Computations in Einsummable".  Citations below name its sections,
 * definitions and examples.
 *
 * Error convention: 0 on success, negative on bad arguments.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define OR_MAX_OPERANDS 9 /* up to 8 inputs + the output */
#define OR_MAX_RANK 8

int or_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads of the parallel loops that follow (n >= 1); timing only. */
void or_set_num_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* ------------------------------------------------------------------------ */
/* Rounding.  fp64 -> bf16 round-to-nearest-even, returned widened to fp64.  */
/* bf16 keeps 8 significant bits; the quantum of a value x = m*2^e with      */
/* m in [0.5,1) is 2^(e-8), and 2^-133 below the normal range (e < -125).    */
/* Values beyond the bf16 range are outside every workload here.             */
/* ------------------------------------------------------------------------ */
static double rne_bf16_one(double x) {
  if (x == 0.0 || isnan(x) || isinf(x)) return x;
  int e;
  frexp(x, &e);
  if (e < -125) e = -125;
  double q = ldexp(1.0, e - 8);
  double t = x / q;           /* exact: division by a power of two */
  double r = nearbyint(t);    /* ties to even under the default mode */
  return r * q;
}

int or_rne_bf16(int64_t n, const double* x, double* y) {
  if (n < 0 || (n > 0 && (!x || !y))) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) y[i] = rne_bf16_one(x[i]);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Block layout of a tensor relation (Section 3.1, tensor types and tilings; */
/* Section 1, a tensor relation is a set of (key, sub-tensor) pairs).        */
/*                                                                           */
/* Partition: per dim d, nblocks[d] intervals given by nblocks[d]+1 split    */
/* points, strictly increasing from 0 to the extent.  Blocks are stored in   */
/* row-major order of their block coordinates; each block is row-major over  */
/* its own extents; every block starts at a multiple of 256 bytes; the      */
/* relation's byte size ends at the last element of the last block.          */
/* ------------------------------------------------------------------------ */
static int check_partition(int rank, const int64_t* nblocks, const int64_t* splits) {
  if (rank < 1 || rank > OR_MAX_RANK || !nblocks || !splits) return -1;
  const int64_t* s = splits;
  for (int d = 0; d < rank; ++d) {
    if (nblocks[d] < 1) return -1;
    if (s[0] != 0) return -1;
    for (int64_t b = 0; b < nblocks[d]; ++b)
      if (s[b + 1] <= s[b]) return -1;
    s += nblocks[d] + 1;
  }
  return 0;
}

/* Per-dim pointer to the split list. */
static void split_ptrs(int rank, const int64_t* nblocks, const int64_t* splits,
                       const int64_t** sp) {
  const int64_t* s = splits;
  for (int d = 0; d < rank; ++d) { sp[d] = s; s += nblocks[d] + 1; }
}

int or_layout(int rank, const int64_t* nblocks, const int64_t* splits,
              int64_t elem_size, int64_t* offsets, int64_t* nbytes) {
  if (check_partition(rank, nblocks, splits) || elem_size <= 0) return -1;
  const int64_t* sp[OR_MAX_RANK];
  split_ptrs(rank, nblocks, splits, sp);
  int64_t nb = 1;
  for (int d = 0; d < rank; ++d) nb *= nblocks[d];
  int64_t c[OR_MAX_RANK] = {0};
  int64_t pos = 0, end = 0;
  for (int64_t b = 0; b < nb; ++b) {
    /* block coordinates of b, row-major over nblocks */
    int64_t rem = b;
    for (int d = rank - 1; d >= 0; --d) { c[d] = rem % nblocks[d]; rem /= nblocks[d]; }
    int64_t n = 1;
    for (int d = 0; d < rank; ++d) n *= sp[d][c[d] + 1] - sp[d][c[d]];
    pos = (pos + 255) / 256 * 256;
    if (offsets) offsets[b] = pos;
    end = pos + n * elem_size;
    pos = end;
  }
  if (nbytes) *nbytes = end;
  return 0;
}

/* Copy between a dense row-major tensor and its block-major relation.
 * to_blocks != 0: dense -> blocked; otherwise blocked -> dense. */
static int pack_impl(int rank, const int64_t* nblocks, const int64_t* splits,
                     int64_t es, const char* src, char* dst, int to_blocks) {
  if (check_partition(rank, nblocks, splits) || es <= 0 || !src || !dst) return -1;
  const int64_t* sp[OR_MAX_RANK];
  split_ptrs(rank, nblocks, splits, sp);
  int64_t shape[OR_MAX_RANK];
  for (int d = 0; d < rank; ++d) shape[d] = sp[d][nblocks[d]];
  int64_t nb = 1;
  for (int d = 0; d < rank; ++d) nb *= nblocks[d];
  int64_t* offs = (int64_t*)malloc(sizeof(int64_t) * nb);
  if (!offs) return -1;
  or_layout(rank, nblocks, splits, es, offs, NULL);
#pragma omp parallel for schedule(dynamic)
  for (int64_t b = 0; b < nb; ++b) {
    int64_t c[OR_MAX_RANK], lo[OR_MAX_RANK], ext[OR_MAX_RANK], r[OR_MAX_RANK];
    int64_t rem = b;
    for (int d = rank - 1; d >= 0; --d) { c[d] = rem % nblocks[d]; rem /= nblocks[d]; }
    int64_t n = 1;
    for (int d = 0; d < rank; ++d) {
      lo[d] = sp[d][c[d]];
      ext[d] = sp[d][c[d] + 1] - lo[d];
      n *= ext[d];
      r[d] = 0;
    }
    for (int64_t e = 0; e < n; ++e) {
      /* dense flat index of block element r (row-major within the block) */
      int64_t flat = 0;
      for (int d = 0; d < rank; ++d) flat = flat * shape[d] + lo[d] + r[d];
      if (to_blocks)
        memcpy(dst + offs[b] + e * es, src + flat * es, (size_t)es);
      else
        memcpy(dst + flat * es, src + offs[b] + e * es, (size_t)es);
      for (int d = rank - 1; d >= 0; --d) {
        if (++r[d] < ext[d]) break;
        r[d] = 0;
      }
    }
  }
  free(offs);
  return 0;
}

int or_pack(int rank, const int64_t* nblocks, const int64_t* splits, int64_t es,
            const void* dense, void* blocked) {
  return pack_impl(rank, nblocks, splits, es, (const char*)dense, (char*)blocked, 1);
}

int or_unpack(int rank, const int64_t* nblocks, const int64_t* splits, int64_t es,
              const void* blocked, void* dense) {
  return pack_impl(rank, nblocks, splits, es, (const char*)blocked, (char*)dense, 0);
}

/* ------------------------------------------------------------------------ */
/* Spec parser: "ij,jk->ik".  Letters a-z and A-Z; every output letter must  */
/* appear in some input; no letter may repeat inside one operand.            */
/* ------------------------------------------------------------------------ */
typedef struct {
  int n_ops;                       /* inputs + 1; the output is last */
  int rank[OR_MAX_OPERANDS];
  char let[OR_MAX_OPERANDS][OR_MAX_RANK];
} or_spec;

static int is_letter(char ch) {
  return (ch >= 'a' && ch <= 'z') || (ch >= 'A' && ch <= 'Z');
}

static int parse_spec(const char* s, or_spec* sp) {
  if (!s) return -1;
  memset(sp, 0, sizeof(*sp));
  const char* arrow = strstr(s, "->");
  if (!arrow) return -1;
  int op = 0, r = 0;
  for (const char* p = s;; ++p) {
    if (p == arrow || *p == ',') {
      if (r == 0 || op >= OR_MAX_OPERANDS - 1) return -1;
      sp->rank[op++] = r;
      r = 0;
      if (p == arrow) break;
      continue;
    }
    if (!is_letter(*p) || r >= OR_MAX_RANK) return -1;
    for (int i = 0; i < r; ++i) if (sp->let[op][i] == *p) return -1;
    sp->let[op][r++] = *p;
  }
  for (const char* p = arrow + 2; *p; ++p) {
    if (!is_letter(*p) || r >= OR_MAX_RANK) return -1;
    for (int i = 0; i < r; ++i) if (sp->let[op][i] == *p) return -1;
    sp->let[op][r++] = *p;
  }
  if (r == 0) return -1;
  sp->rank[op] = r;
  sp->n_ops = op + 1;
  /* every output letter must come from an input */
  for (int i = 0; i < r; ++i) {
    int found = 0;
    for (int o = 0; o < op && !found; ++o)
      for (int j = 0; j < sp->rank[o]; ++j) if (sp->let[o][j] == sp->let[op][i]) found = 1;
    if (!found) return -1;
  }
  return 0;
}

static int find_dim(const or_spec* sp, int op, char l) {
  for (int i = 0; i < sp->rank[op]; ++i) if (sp->let[op][i] == l) return i;
  return -1;
}

/* ------------------------------------------------------------------------ */
/* Join (Section 3.2, Definitions "Join-agg spec" and "Implementation",      */
/* step 1; Section 3.3 for the count of function specifications).           */
/*                                                                           */
/* Brute force: every combination of one block per input is tested; it is   */
/* kept iff each letter shared by two or more inputs has the identical       */
/* interval (lo, hi) in each of them, and, when a causal pair of letters     */
/* (q, k) is given, iff the k block starts at or before the last q row       */
/* (k_lo <= q_hi - 1).  Each kept tuple records the output block whose       */
/* intervals on the output letters equal the tuple's.                        */
/*                                                                           */
/* Order: tuples are grouped by the block coordinates of the `group` letters */
/* (row-major, in the order they are listed), and inside a group ordered by  */
/* the block coordinates of the remaining letters in order of first          */
/* appearance across the inputs.  group_off is the CSR offset array over all */
/* group-letter block combinations (empty groups included).                  */
/*                                                                           */
/* Operand partitions: nblocks_all holds rank entries per operand (inputs,   */
/* then output); splits_all holds, per operand and per dim, nblocks+1 split  */
/* points.  Returns the tuple count, or a negative error:                    */
/*   -1 bad arguments, -2 output partition lacks a tuple's interval,         */
/*   -3 capacity too small.                                                  */
/* ------------------------------------------------------------------------ */
typedef struct {
  int64_t sort_key[2 * OR_MAX_RANK + 2];
  int nkey;
  int32_t rec[OR_MAX_OPERANDS];
} or_tuple;

static int tuple_cmp(const void* a, const void* b) {
  const or_tuple* x = (const or_tuple*)a;
  const or_tuple* y = (const or_tuple*)b;
  for (int i = 0; i < x->nkey; ++i) {
    if (x->sort_key[i] < y->sort_key[i]) return -1;
    if (x->sort_key[i] > y->sort_key[i]) return 1;
  }
  return 0;
}

/* Sequence of position x among packed sequences ending at ends[0..n): the
   number of ends at or below x (Section 3.3, Example "Flash attention"). */
static int64_t seq_index(const int64_t* ends, int64_t n, int64_t x) {
  int64_t s = 0;
  while (s < n && ends[s] <= x) ++s;
  return s;
}

/* Attention visibility of key position kp to query position qp: the same
   sequence (when sequences are given) and, when causal, kp <= qp. */
static int visible(int64_t qp, int64_t kp, int causal, const int64_t* ends, int64_t n_seq) {
  if (causal && kp > qp) return 0;
  if (n_seq > 0 && seq_index(ends, n_seq, qp) != seq_index(ends, n_seq, kp)) return 0;
  return 1;
}

int64_t or_join_ex(const char* spec, const int64_t* nblocks_all, const int64_t* splits_all,
                   const char* group, char pos_q, char pos_k, int causal, int64_t n_seq,
                   const int64_t* seq_ends, int64_t gqa, char gqa_h, char gqa_g,
                   int32_t* tuples, int64_t cap, int64_t* group_off, int64_t gcap,
                   int64_t* n_groups_out);

/* The plain join: causal_q/causal_k (0 = none) name the letters of the
   causal predicate. */
int64_t or_join(const char* spec, const int64_t* nblocks_all, const int64_t* splits_all,
                const char* group, char causal_q, char causal_k,
                int32_t* tuples, int64_t cap, int64_t* group_off, int64_t gcap,
                int64_t* n_groups_out) {
  return or_join_ex(spec, nblocks_all, splits_all, group, causal_q, causal_k, causal_q != 0, 0, NULL, 1, 0, 0,
                    tuples, cap, group_off, gcap, n_groups_out);
}

/* The join with attention's predicates.  pos_q/pos_k name the query and key
   position letters (0: no position predicate).  A tuple is kept iff some
   query position of its query block sees some key position of its key block
   (visible() above: causal order if `causal`, and with n_seq > 0 packed
   sequences the same sequence).  gqa > 1: grouped-query heads, letter gqa_h
   (query heads) over gqa_g (key/value heads); a tuple is kept iff every
   query head h of its gqa_h block reads key/value head floor(h / gqa),
   inside its gqa_g block. */
int64_t or_join_ex(const char* spec, const int64_t* nblocks_all, const int64_t* splits_all,
                   const char* group, char pos_q, char pos_k, int causal, int64_t n_seq,
                   const int64_t* seq_ends, int64_t gqa, char gqa_h, char gqa_g,
                   int32_t* tuples, int64_t cap, int64_t* group_off, int64_t gcap,
                   int64_t* n_groups_out) {
  const char causal_q = pos_q, causal_k = pos_k;
  if ((causal || n_seq > 0) && !pos_q) return -1;
  if (n_seq < 0 || (n_seq > 0 && !seq_ends) || gqa < 1 || (gqa > 1 && (!gqa_h || !gqa_g))) return -1;
  or_spec sp;
  if (parse_spec(spec, &sp) || !nblocks_all || !splits_all || !group) return -1;
  const int n_in = sp.n_ops - 1, out = n_in;
  /* per operand, per dim: nblocks and split pointers */
  const int64_t* nbk[OR_MAX_OPERANDS];
  const int64_t* spl[OR_MAX_OPERANDS][OR_MAX_RANK];
  int64_t nb_tot[OR_MAX_OPERANDS];
  {
    const int64_t* nbp = nblocks_all;
    const int64_t* spp = splits_all;
    for (int o = 0; o < sp.n_ops; ++o) {
      if (check_partition(sp.rank[o], nbp, spp)) return -1;
      nbk[o] = nbp;
      nb_tot[o] = 1;
      for (int d = 0; d < sp.rank[o]; ++d) {
        spl[o][d] = spp;
        spp += nbp[d] + 1;
        nb_tot[o] *= nbp[d];
      }
      nbp += sp.rank[o];
    }
  }
  /* group letters must be output letters */
  int ng_let = (int)strlen(group);
  if (ng_let > OR_MAX_RANK) return -1;
  int64_t n_groups = 1;
  int g_dim[OR_MAX_RANK];
  for (int i = 0; i < ng_let; ++i) {
    g_dim[i] = find_dim(&sp, out, group[i]);
    if (g_dim[i] < 0) return -1;
    n_groups *= nbk[out][g_dim[i]];
  }
  /* remaining letters in order of first appearance across the inputs */
  char rest[OR_MAX_OPERANDS * OR_MAX_RANK];
  int n_rest = 0;
  for (int o = 0; o < n_in; ++o)
    for (int d = 0; d < sp.rank[o]; ++d) {
      char l = sp.let[o][d];
      if (memchr(group, l, (size_t)ng_let)) continue;
      if (n_rest && memchr(rest, l, (size_t)n_rest)) continue;
      rest[n_rest++] = l;
    }
  /* causal letters: the operands that carry them */
  int cq_op = -1, cq_dim = -1, ck_op = -1, ck_dim = -1;
  if (causal_q) {
    for (int o = 0; o < n_in && cq_op < 0; ++o)
      if ((cq_dim = find_dim(&sp, o, causal_q)) >= 0) cq_op = o;
    for (int o = 0; o < n_in && ck_op < 0; ++o)
      if ((ck_dim = find_dim(&sp, o, causal_k)) >= 0) ck_op = o;
    if (cq_op < 0 || ck_op < 0) return -1;
  }
  /* grouped-query head letters */
  int gh_op = -1, gh_dim = -1, gg_op = -1, gg_dim = -1;
  if (gqa > 1) {
    for (int o = 0; o < n_in && gh_op < 0; ++o)
      if ((gh_dim = find_dim(&sp, o, gqa_h)) >= 0) gh_op = o;
    for (int o = 0; o < n_in && gg_op < 0; ++o)
      if ((gg_dim = find_dim(&sp, o, gqa_g)) >= 0) gg_op = o;
    if (gh_op < 0 || gg_op < 0) return -1;
  }

  int64_t n_comb = 1;
  for (int o = 0; o < n_in; ++o) n_comb *= nb_tot[o];
  or_tuple* kept = (or_tuple*)malloc(sizeof(or_tuple) * (size_t)(n_comb > 0 ? n_comb : 1));
  if (!kept) return -1;
  int64_t n_kept = 0;
  int err = 0;

  int64_t bidx[OR_MAX_OPERANDS] = {0};
  for (int64_t comb = 0; comb < n_comb && !err; ++comb) {
    int64_t rem = comb;
    for (int o = n_in - 1; o >= 0; --o) { bidx[o] = rem % nb_tot[o]; rem /= nb_tot[o]; }
    /* block coordinates and intervals of each input block */
    int64_t lo[OR_MAX_OPERANDS][OR_MAX_RANK], hi[OR_MAX_OPERANDS][OR_MAX_RANK];
    int64_t bc[OR_MAX_OPERANDS][OR_MAX_RANK];
    for (int o = 0; o < n_in; ++o) {
      int64_t r2 = bidx[o];
      for (int d = sp.rank[o] - 1; d >= 0; --d) {
        bc[o][d] = r2 % nbk[o][d];
        r2 /= nbk[o][d];
        lo[o][d] = spl[o][d][bc[o][d]];
        hi[o][d] = spl[o][d][bc[o][d] + 1];
      }
    }
    /* join condition: identical intervals on every shared letter */
    int ok = 1;
    for (int o = 0; o < n_in && ok; ++o)
      for (int d = 0; d < sp.rank[o] && ok; ++d)
        for (int o2 = o + 1; o2 < n_in && ok; ++o2) {
          int d2 = find_dim(&sp, o2, sp.let[o][d]);
          if (d2 >= 0 && (lo[o2][d2] != lo[o][d] || hi[o2][d2] != hi[o][d])) ok = 0;
        }
    if (!ok) continue;
    if (causal_q && (causal || n_seq > 0)) {
      int any = 0;
      for (int64_t qp = lo[cq_op][cq_dim]; qp < hi[cq_op][cq_dim] && !any; ++qp)
        for (int64_t kp = lo[ck_op][ck_dim]; kp < hi[ck_op][ck_dim] && !any; ++kp)
          any = visible(qp, kp, causal, seq_ends, n_seq);
      if (!any) continue;
    }
    if (gqa > 1) {
      int all = 1;
      for (int64_t h = lo[gh_op][gh_dim]; h < hi[gh_op][gh_dim] && all; ++h)
        all = h / gqa >= lo[gg_op][gg_dim] && h / gqa < hi[gg_op][gg_dim];
      if (!all) continue;
    }
    /* output block: the one whose intervals equal the tuple's on every output letter */
    or_tuple t;
    memset(&t, 0, sizeof(t));
    int64_t ob = 0, oc[OR_MAX_RANK];
    for (int d = 0; d < sp.rank[out] && !err; ++d) {
      char l = sp.let[out][d];
      int64_t l_lo = -1, l_hi = -1;
      for (int o = 0; o < n_in && l_lo < 0; ++o) {
        int dd = find_dim(&sp, o, l);
        if (dd >= 0) { l_lo = lo[o][dd]; l_hi = hi[o][dd]; }
      }
      int64_t found = -1;
      for (int64_t b = 0; b < nbk[out][d]; ++b)
        if (spl[out][d][b] == l_lo && spl[out][d][b + 1] == l_hi) found = b;
      if (found < 0) { err = -2; break; }
      oc[d] = found;
      ob = ob * nbk[out][d] + found;
    }
    if (err) break;
    t.rec[0] = (int32_t)ob;
    for (int o = 0; o < n_in; ++o) t.rec[1 + o] = (int32_t)bidx[o];
    /* sort key: group-letter block coordinates, then the rest */
    int64_t gkey = 0;
    for (int i = 0; i < ng_let; ++i) gkey = gkey * nbk[out][g_dim[i]] + oc[g_dim[i]];
    t.sort_key[t.nkey++] = gkey;
    for (int i = 0; i < n_rest; ++i) {
      int64_t lo_l = -1;
      for (int o = 0; o < n_in && lo_l < 0; ++o) {
        int dd = find_dim(&sp, o, rest[i]);
        if (dd >= 0) lo_l = lo[o][dd];
      }
      t.sort_key[t.nkey++] = lo_l;
    }
    kept[n_kept++] = t;
  }
  if (err) { free(kept); return err; }
  qsort(kept, (size_t)n_kept, sizeof(or_tuple), tuple_cmp);
  if (n_groups_out) *n_groups_out = n_groups;
  if (tuples && n_kept > cap) { free(kept); return -3; }
  if (group_off && n_groups + 1 > gcap) { free(kept); return -3; }
  if (tuples)
    for (int64_t i = 0; i < n_kept; ++i)
      for (int o = 0; o <= n_in; ++o) tuples[i * (n_in + 1) + o] = kept[i].rec[o];
  if (group_off) {
    int64_t i = 0;
    for (int64_t g = 0; g <= n_groups; ++g) {
      while (i < n_kept && kept[i].sort_key[0] < g) ++i;
      group_off[g] = i;
    }
  }
  free(kept);
  return n_kept;
}

/* ------------------------------------------------------------------------ */
/* Generic dense einsum with a join operation and an aggregation             */
/* (Section 3.2, Definition "Implementation", taken densely: in the          */
/* degenerate relation of Section 1 each key is one cell, each sub-tensor a  */
/* scalar, and a join-agg is a join on the shared indices plus a GROUP BY    */
/* over the output indices).                                                 */
/*   out[o] = AGG over all values c of the contracted letters of             */
/*            JOIN(in_1[..], ..., in_n[..])                                  */
/* JOIN: 0 = product of the inputs, 1 = sum of the inputs.                   */
/* AGG:  0 = none (no contracted letters allowed), 1 = sum (identity 0),     */
/*       2 = max (identity -inf).                                            */
/* shapes_all: rank entries per operand, inputs then output.                 */
/* ------------------------------------------------------------------------ */
int or_einsum(const char* spec, int join_op, int agg_op, const int64_t* shapes_all,
              const double* const* ins, double* out) {
  or_spec sp;
  if (parse_spec(spec, &sp) || !shapes_all || !ins || !out) return -1;
  if (join_op < 0 || join_op > 1 || agg_op < 0 || agg_op > 2) return -1;
  const int n_in = sp.n_ops - 1, oo = n_in;
  /* letter sizes, consistent across operands */
  char letters[64];
  int64_t lsize[64];
  int nl = 0;
  const int64_t* shp[OR_MAX_OPERANDS];
  {
    const int64_t* p = shapes_all;
    for (int o = 0; o < sp.n_ops; ++o) { shp[o] = p; p += sp.rank[o]; }
  }
  for (int o = 0; o < sp.n_ops; ++o)
    for (int d = 0; d < sp.rank[o]; ++d) {
      char l = sp.let[o][d];
      int i;
      for (i = 0; i < nl; ++i) if (letters[i] == l) break;
      if (i == nl) { letters[nl] = l; lsize[nl] = shp[o][d]; ++nl; }
      else if (lsize[i] != shp[o][d]) return -1;
      if (shp[o][d] < 1) return -1;
    }
  /* contracted letters: in some input, not in the output */
  int ci[64], nc = 0;
  int64_t n_contr = 1;
  for (int i = 0; i < nl; ++i)
    if (find_dim(&sp, oo, letters[i]) < 0) { ci[nc++] = i; n_contr *= lsize[i]; }
  if (agg_op == 0 && nc > 0) return -1;
  int oi[OR_MAX_RANK];
  int64_t n_out = 1;
  for (int d = 0; d < sp.rank[oo]; ++d) {
    for (int i = 0; i < nl; ++i) if (letters[i] == sp.let[oo][d]) oi[d] = i;
    n_out *= shp[oo][d];
  }
  /* per input, letter index of each dim */
  int li[OR_MAX_OPERANDS][OR_MAX_RANK];
  for (int o = 0; o < n_in; ++o)
    for (int d = 0; d < sp.rank[o]; ++d)
      for (int i = 0; i < nl; ++i) if (letters[i] == sp.let[o][d]) li[o][d] = i;

#pragma omp parallel for schedule(static)
  for (int64_t flat = 0; flat < n_out; ++flat) {
    int64_t val[64];
    int64_t rem = flat;
    for (int d = sp.rank[oo] - 1; d >= 0; --d) {
      val[oi[d]] = rem % shp[oo][d];
      rem /= shp[oo][d];
    }
    double acc = agg_op == 2 ? -INFINITY : 0.0;
    for (int64_t c = 0; c < n_contr; ++c) {
      int64_t r2 = c;
      for (int j = nc - 1; j >= 0; --j) { val[ci[j]] = r2 % lsize[ci[j]]; r2 /= lsize[ci[j]]; }
      double f = join_op == 0 ? 1.0 : 0.0;
      for (int o = 0; o < n_in; ++o) {
        int64_t idx = 0;
        for (int d = 0; d < sp.rank[o]; ++d) idx = idx * shp[o][d] + val[li[o][d]];
        f = join_op == 0 ? f * ins[o][idx] : f + ins[o][idx];
      }
      if (agg_op == 2) acc = f > acc ? f : acc;
      else if (agg_op == 1) acc += f;
      else acc = f;
    }
    out[flat] = acc;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Dense matrix product C[M,N] = A[M,K] * B[K,N], fp64, the textbook triple  */
/* loop (Section 3.2, Examples "Matrix multiply" as the abstract operator).  */
/* ------------------------------------------------------------------------ */
int or_matmul(int64_t M, int64_t K, int64_t N, const double* A, const double* B, double* C) {
  if (M < 1 || K < 1 || N < 1 || !A || !B || !C) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < M; ++i) {
    double* c = C + i * N;
    for (int64_t j = 0; j < N; ++j) c[j] = 0.0;
    for (int64_t k = 0; k < K; ++k) {
      const double a = A[i * K + k];
      const double* b = B + k * N;
      for (int64_t j = 0; j < N; ++j) c[j] += a * b[j];
    }
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* RMS normalisation of each row of x[T,C] (the paper lists normalisation    */
/* among the operators that are a join followed by an aggregation, Section   */
/* 1; its formula is not given there, so the LLaMA convention is used):      */
/*   y[t,c] = w[c] * x[t,c] / sqrt( (1/C) * sum_c' x[t,c']^2 + eps )         */
/* ------------------------------------------------------------------------ */
int or_rmsnorm(int64_t T, int64_t C, const double* x, const double* w, double eps, double* y) {
  if (T < 1 || C < 1 || !x || !w || !y) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < T; ++t) {
    const double* xr = x + t * C;
    double ss = 0.0;
    for (int64_t c = 0; c < C; ++c) ss += xr[c] * xr[c];
    double inv = 1.0 / sqrt(ss / (double)C + eps);
    for (int64_t c = 0; c < C; ++c) y[t * C + c] = w[c] * xr[c] * inv;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Row softmax of s[H,Q,K] over its last index, two passes (max, then the    */
/* sum of exponentials).  With causal != 0, key k is visible to query q iff  */
/* k <= q; invisible entries get probability exactly 0.                      */
/* ------------------------------------------------------------------------ */
int or_softmax(int64_t H, int64_t Q, int64_t K, const double* s, int causal, double* p) {
  if (H < 1 || Q < 1 || K < 1 || !s || !p) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t hq = 0; hq < H * Q; ++hq) {
    const int64_t q = hq % Q;
    const double* sr = s + hq * K;
    double* pr = p + hq * K;
    const int64_t kend = causal ? (q + 1 < K ? q + 1 : K) : K;
    double m = -INFINITY;
    for (int64_t k = 0; k < kend; ++k) m = sr[k] > m ? sr[k] : m;
    double l = 0.0;
    for (int64_t k = 0; k < kend; ++k) l += exp(sr[k] - m);
    for (int64_t k = 0; k < K; ++k) pr[k] = k < kend ? exp(sr[k] - m) / l : 0.0;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Scaled dot-product attention per (batch, head), q[B,H,S,D], k and v       */
/* [B,H,S,D], out o[B,H,S,D] (Section 3.3, Example "Flash attention" names   */
/* the operator; the causal rule and the scale are stated readings):         */
/*   s[q,k] = scale * sum_d q[q,d] k[k,d];  p = softmax over visible k;       */
/*   o[q,d] = sum_k p[q,k] v[k,d].  Causal: k visible to q iff k <= q.       */
/* ------------------------------------------------------------------------ */
int or_attention(int64_t B, int64_t H, int64_t S, int64_t D, const double* q,
                 const double* k, const double* v, int causal, double scale, double* o) {
  if (B < 1 || H < 1 || S < 1 || D < 1 || !q || !k || !v || !o) return -1;
#pragma omp parallel
  {
    double* srow = (double*)malloc(sizeof(double) * (size_t)S);
#pragma omp for schedule(dynamic, 4)
    for (int64_t r = 0; r < B * H * S; ++r) {
      const int64_t bh = r / S, qi = r % S;
      const double* qr = q + r * D;
      const double* kb = k + bh * S * D;
      const double* vb = v + bh * S * D;
      const int64_t kend = causal ? qi + 1 : S;
      double m = -INFINITY;
      for (int64_t j = 0; j < kend; ++j) {
        double acc = 0.0;
        for (int64_t d = 0; d < D; ++d) acc += qr[d] * kb[j * D + d];
        srow[j] = scale * acc;
        m = srow[j] > m ? srow[j] : m;
      }
      double l = 0.0;
      for (int64_t j = 0; j < kend; ++j) { srow[j] = exp(srow[j] - m); l += srow[j]; }
      double* orow = o + r * D;
      for (int64_t d = 0; d < D; ++d) orow[d] = 0.0;
      for (int64_t j = 0; j < kend; ++j) {
        const double pj = srow[j] / l;
        for (int64_t d = 0; d < D; ++d) orow[d] += pj * vb[j * D + d];
      }
    }
    free(srow);
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Attention with grouped-query heads and packed sequences (Section 3.2,     */
/* Example "Flash attention"): q [B, Hq, S, D], k and v [B, Hkv, S, D] with   */
/* Hq a multiple of Hkv; query head h reads key/value head h / (Hq / Hkv).   */
/* The sequence axis holds n_seq sequences ending at seq_ends (n_seq 0: one  */
/* sequence).  Query qi sees key j iff visible(qi, j): same sequence and,    */
/* if causal, j <= qi.  s = scale * q.k; o = softmax over the visible keys   */
/* of s, times v.  A row with no visible key (impossible for the causal or   */
/* packed rules, which keep j = qi) is 0.                                    */
/* ------------------------------------------------------------------------ */
int or_attention_ex(int64_t B, int64_t Hq, int64_t Hkv, int64_t S, int64_t D, const double* q,
                    const double* k, const double* v, int causal, double scale, int64_t n_seq,
                    const int64_t* seq_ends, double* o) {
  if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || S < 1 || D < 1 || !q || !k || !v || !o) return -1;
  if (n_seq < 0 || (n_seq > 0 && (!seq_ends || seq_ends[n_seq - 1] != S))) return -1;
  const int64_t G = Hq / Hkv;
#pragma omp parallel
  {
    double* srow = (double*)malloc(sizeof(double) * (size_t)S);
    char* vis = (char*)malloc((size_t)S);
#pragma omp for schedule(dynamic, 4)
    for (int64_t r = 0; r < B * Hq * S; ++r) {
      const int64_t b = r / (Hq * S), h = (r / S) % Hq, qi = r % S;
      const double* qr = q + r * D;
      const double* kb = k + (b * Hkv + h / G) * S * D;
      const double* vb = v + (b * Hkv + h / G) * S * D;
      double m = -INFINITY;
      for (int64_t j = 0; j < S; ++j) {
        vis[j] = (char)visible(qi, j, causal, seq_ends, n_seq);
        if (!vis[j]) continue;
        double acc = 0.0;
        for (int64_t d = 0; d < D; ++d) acc += qr[d] * kb[j * D + d];
        srow[j] = scale * acc;
        m = srow[j] > m ? srow[j] : m;
      }
      double l = 0.0;
      for (int64_t j = 0; j < S; ++j)
        if (vis[j]) { srow[j] = exp(srow[j] - m); l += srow[j]; }
      double* orow = o + r * D;
      for (int64_t d = 0; d < D; ++d) orow[d] = 0.0;
      for (int64_t j = 0; j < S && l > 0.0; ++j) {
        if (!vis[j]) continue;
        const double pj = srow[j] / l;
        for (int64_t d = 0; d < D; ++d) orow[d] += pj * vb[j * D + d];
      }
    }
    free(srow);
    free(vis);
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Elementwise helpers used by the LLaMA-shaped block chain.                 */
/*   silu(g) * u with silu(g) = g / (1 + exp(-g)); and a + b.                */
/* ------------------------------------------------------------------------ */
int or_silu_mul(int64_t n, const double* g, const double* u, double* y) {
  if (n < 0 || (n > 0 && (!g || !u || !y))) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) y[i] = g[i] / (1.0 + exp(-g[i])) * u[i];
  return 0;
}

int or_add(int64_t n, const double* a, const double* b, double* y) {
  if (n < 0 || (n > 0 && (!a || !b || !y))) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) y[i] = a[i] + b[i];
  return 0;
}
