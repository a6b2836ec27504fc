/*
 * ea.h -- C ABI of libea, one GPU's share of a block join-agg on AMD MI355X
 * (gfx950).
 *
 * Model (paper: "Every Kernel Is a Join: Automatic Multi-GPU Parallelism for
 * AI Computations in Einsummable"):
 *  - A tensor relation is a set of (sub_tensor_key, sub_tensor) pairs
 *    (Section 1).  Here a relation is a dense zero-bounded tensor type
 *    (Section 3.1, Definition "Tensor type") cut by a block partition whose
 *    blocks tile it (Section 3.1, Definition "Tiling").  A block's key is its
 *    per-dim block index; its sub-tensor type is (lo, hi) per dim.
 *  - An operation runs as the three steps of Section 3.2, Definition
 *    "Implementation": Join (tuples of one block per input whose shared
 *    einsum letters have identical intervals, each tuple fed to a concrete
 *    per-tuple kernel), Aggregate (tuple results with the same output key
 *    combined by an associative, commutative operator), Recompose (each
 *    aggregated block stored into its slot of the output relation).
 *  - A repartition re-blocks a relation through the overlay of both
 *    partitions (Section 5.3: atoms, decompose and recompose kernels).
 *
 * Memory.  Relation data live in caller-owned device memory (for example a
 * torch uint8 tensor).  Handles hold only host metadata and never free data.
 * Block layout: blocks in row-major order of their block coordinates; each
 * block row-major (C order) over its own extents; each block starts at a
 * multiple of 256 bytes from the relation's base; the relation's size ends at
 * the last element of the last block (ea_layout_nbytes).  Padding bytes are
 * never read for results and never written.
 *
 * Plans.  A join is resolved once per configuration -- spec, ops, dtypes,
 * partitions and parameters, not data pointers -- into a plan: library-owned
 * device tables (block tables, the GPU-built tuple table, the kernel's work
 * list).  Plans are built only by the planning calls ea_joinagg_workspace,
 * ea_repartition_plan and ea_join_tuples: they allocate the plan's device
 * memory, run the GPU join enumerator on the given stream (for block GEMMs and
 * attention, then a kernel that resolves the join into the work list) and
 * wait for it.
 * ea_joinagg and ea_repartition never allocate and never synchronize: they
 * find the plan (EA_ERR_NOPLAN if none was built on the current device) and
 * enqueue kernels.  A plan is immutable once built, so calls that share one
 * may run concurrently on different streams.  Plans live until
 * ea_plan_cache_clear() or process exit.
 *
 * Workspace.  Key-split join-aggs (a block GEMM or attention whose output
 * tiles are cut into several runs of tuples to fill the GPU) exchange partial
 * results through a caller-owned device workspace, of the size that
 * ea_joinagg_workspace reports (0: none needed).  Its first
 * EA_WS_COUNTER_BYTES bytes hold arrival counters: they must be zero before
 * the workspace's first use (allocate it zeroed), and every call leaves them
 * zero again, so one workspace serves any sequence of calls, of any
 * configuration, on one stream.  The bytes after them hold partial results and
 * need no initial value.  Calls that may overlap in time (different streams)
 * need different workspaces.
 *
 * Streams are hipStream_t passed as void*; NULL is the default stream.
 *
 * Errors.  Every call returns EA_OK (0) or a negative EA_ERR_* code and sets a
 * thread-local message (ea_last_error).  No exception crosses the ABI.
 * Argument, spec, partition and join validation runs on the host before any
 * HIP call, so it works without a GPU.  Kernel faults surface as EA_ERR_HIP at
 * the call that observes them.
 */
#ifndef EA_H
#define EA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define EA_VERSION 1
#define EA_MAX_RANK 8
#define EA_MAX_INPUTS 4

/* ---- return codes ---------------------------------------------------- */
#define EA_OK 0
#define EA_ERR_ARG (-1)         /* NULL pointer, bad rank/size/enum value     */
#define EA_ERR_DTYPE (-2)       /* dtype not supported for this operation     */
#define EA_ERR_PARTITION (-3)   /* split points do not tile the shape         */
#define EA_ERR_CAPACITY (-4)    /* buffer smaller than the layout / table     */
#define EA_ERR_SPEC (-5)        /* einsum spec malformed or not matching      */
#define EA_ERR_JOIN (-6)        /* shared letter split differently, or output */
                                /* partition not the one the inputs induce    */
#define EA_ERR_UNSUPPORTED (-7) /* valid request outside what is implemented  */
#define EA_ERR_HIP (-8)         /* a HIP runtime call or kernel failed        */
#define EA_ERR_NOPLAN (-9)      /* configuration not planned on this device:  */
                                /* call the planning entry point first        */

/* Bytes at the start of a join-agg workspace that hold arrival counters. */
#define EA_WS_COUNTER_BYTES 262144

/* ---- element types --------------------------------------------------- */
#define EA_F32 0
#define EA_BF16 1
#define EA_F16 2

/* ---- join operations (the concrete operator f run on each tuple) ------ */
/* Generic einsum join: the scalar join of the inputs' elements.            */
#define EA_JOIN_MUL 0  /* product of the inputs (plain einsum)              */
#define EA_JOIN_ADD 1  /* sum of the inputs                                 */
/* Fused operators (each a join-agg with a fixed spec shape):               */
#define EA_OP_RMSNORM 16   /* "<r>c,c-><r>c": y = w*x/sqrt(mean_c x^2 + eps) */
#define EA_OP_SOFTMAX 17   /* "<r>k-><r>k": softmax over the last letter      */
#define EA_OP_ATTENTION 18 /* "<b>qd,<b>kd,<b>kd-><b>qd": softmax(s*QK^T) V;
                              grouped-query: see ea_params.gqa_group       */
#define EA_OP_SWIGLU 19    /* "tj,jk,jk->tk": silu(X W1) * (X W2)              */

/* ---- aggregation operations (the combiner of tuples sharing a key) ---- */
#define EA_AGG_NONE 0 /* no aggregation: at most one tuple per output key    */
#define EA_AGG_SUM 1  /* addition, identity 0                                */
#define EA_AGG_MAX 2  /* maximum, identity -inf                              */
#define EA_AGG_LSE 3  /* online softmax: (m, l, O) pairs combined by
                         m = max(m1, m2), l = l1 e^(m1-m) + l2 e^(m2-m),
                         O = O1 e^(m1-m) + O2 e^(m2-m)                       */

typedef struct ea_relation ea_relation;

/* Per-call parameters.  Zero-initialise and set what the operation uses. */
/* Output store policy (ea_params.store, ea_repartition_ex).  CACHED: plain
   stores; the output stays in the GPU's caches for a kernel that reads it
   next.  STREAM: non-temporal stores; the output is streamed towards memory,
   which suits an output that nothing reads soon or that exceeds the caches
   (the end of a kernel then has no dirty cache lines of it to write back).
   Results are bit-identical under both. */
#define EA_STORE_CACHED 0
#define EA_STORE_STREAM 1

typedef struct ea_params {
  float eps;    /* EA_OP_RMSNORM: added to the mean square (e.g. 1e-6)       */
  float scale;  /* EA_OP_ATTENTION: multiplier of the q.k scores (> 0)       */
  int32_t causal; /* EA_OP_SOFTMAX / EA_OP_ATTENTION: 1 = key position k is
                     visible to query position q iff k <= q (0-based)        */
  int32_t store;  /* EA_STORE_CACHED (0, default) or EA_STORE_STREAM (1);
                     honoured by EA_OP_RMSNORM and EA_OP_SOFTMAX (the block
                     GEMM, attention and general einsum paths store plainly,
                     their outputs feeding the next operator).  Other
                     values: EA_ERR_ARG.                                     */
  /* Optional relation added to the aggregated result before the store
     (fused residual): same shape and partition as the output.  Used by the
     einsum path (EA_JOIN_MUL / EA_JOIN_ADD).  NULL = none.                  */
  const ea_relation* residual;
  /* EA_OP_ATTENTION, grouped-query attention (Section 3.3, Example "Flash
     attention"): query heads per key-value head.  0 or 1: Q, K and V share
     every batch letter.  G > 1: K and V name their head letter apart from
     Q's ("bhqd,bgkd,bgkd->bhqd"), Q's head extent is G times theirs, and
     query head h reads key-value head floor(h / G); the join keeps a tuple
     iff the K/V head block holds the heads of the Q head block divided by G.
     Head letters take one block per index.  Negative: EA_ERR_ARG.           */
  int32_t gqa_group;
  /* EA_OP_ATTENTION, packed sequences (same example): the query/key letter
     holds n_seq independent sequences end to end, ending at the host array
     seq_ends[0..n_seq) (strictly increasing, the last equal to the extent,
     read during the call only).  A query attends only to keys of its own
     sequence (and, if causal, at or before its position); the join keeps a
     query block and a key block iff they lie in the same sequence.  Every
     end must be a split point of the query and of the key partition: no
     block straddles two sequences (EA_ERR_UNSUPPORTED otherwise).  n_seq 0:
     one sequence; seq_ends NULL with n_seq > 0, or a bad list: EA_ERR_ARG.  */
  int32_t n_seq;
  const int64_t* seq_ends;
} ea_params;

/* ---- version and errors ---------------------------------------------- */
int ea_version(void);
/* Message for the last non-zero return on this thread ("" if none).  The
   pointer stays valid until the next ea_* call on the same thread. */
const char* ea_last_error(void);
/* Bytes per element of a dtype, or EA_ERR_DTYPE. */
int ea_dtype_size(int32_t dtype);

/* ---- layout and relations (Section 3.1) ------------------------------- */
/* Bytes a relation of this shape, dtype and partition occupies.
   rank in [1, 8]; shape[d] >= 1; nblocks[d] >= 1; splits concatenates, per
   dim, nblocks[d]+1 strictly increasing points from 0 to shape[d].
   Errors: EA_ERR_ARG, EA_ERR_DTYPE, EA_ERR_PARTITION. */
int ea_layout_nbytes(int32_t rank, const int64_t* shape, int32_t dtype,
                     const int32_t* nblocks, const int64_t* splits, int64_t* nbytes);

/* Create a relation handle over caller-owned device memory.
   data: base of the block-major storage (may be NULL for metadata-only use;
   compute calls then fail with EA_ERR_ARG); capacity: its size in bytes,
   >= ea_layout_nbytes unless data is NULL.  Arrays are copied.
   Errors: EA_ERR_ARG, EA_ERR_DTYPE, EA_ERR_PARTITION, EA_ERR_CAPACITY. */
int ea_relation_create(int32_t rank, const int64_t* shape, int32_t dtype,
                       const int32_t* nblocks, const int64_t* splits,
                       void* data, int64_t capacity, ea_relation** out);
/* Free the handle (never the data).  NULL is accepted and ignored. */
int ea_relation_destroy(ea_relation* rel);
/* Re-point a relation at other memory of at least its layout's size. */
int ea_relation_set_data(ea_relation* rel, void* data, int64_t capacity);
int ea_relation_num_blocks(const ea_relation* rel, int64_t* n);
int ea_relation_nbytes(const ea_relation* rel, int64_t* nbytes);
/* Block b's key as its sub-tensor type: lo[d] inclusive, hi[d] exclusive
   (arrays of the relation's rank), and its byte offset from the base. */
int ea_relation_block(const ea_relation* rel, int64_t b, int64_t* lo, int64_t* hi,
                      int64_t* byte_off);

/* ---- join-agg (Section 3.2, Definitions "Join-agg spec", "Implementation")
   spec: explicit einsum "ij,jk->ik" over letters a-z/A-Z.  in[i] takes the
   letters of the i-th operand; out the letters after "->".  Every letter
   shared by two or more operands must have the same extent and the same
   split points in each (EA_ERR_JOIN otherwise: repartition first); the
   output's partition on each letter must equal the inputs' (EA_ERR_JOIN).
   Tuples are grouped by output key; inside a group they are combined by
   agg_op in ascending order of the contracted letters' blocks, so results
   are deterministic (no atomics in the combine).

   join_op EA_JOIN_MUL / EA_JOIN_ADD, agg_op NONE / SUM / MAX: out[o] =
     AGG over contracted letter values of JOIN(in_1[..], ..., in_n[..]),
     then + residual if given.  NONE requires no contracted letters.  Inputs
     and output f32, bf16 or f16; arithmetic in f32.  A two-operand product
     "ab,bc->ac" or "ab,cb->ac" with bf16 inputs runs on the bf16 matrix
     cores (fp32 accumulation).
   EA_OP_RMSNORM, agg SUM: in = (x "<r>c", w "c"); out "<r>c" with x's
     letters; y = w * x / sqrt(sum_c x^2 / C + eps) over the full extent C
     of the last letter (params->eps).  The sum of squares is aggregated
     over all blocks of c.  bf16/f32 data, f32 arithmetic.
   EA_OP_SOFTMAX, agg LSE: in = s "<r>k" (rank >= 2 if causal), out with the
     same letters; softmax over the last letter; with params->causal the
     second-to-last letter is the query position and invisible entries are 0.
   EA_OP_ATTENTION, agg LSE: in = (Q "<b>qd", K "<b>kd", V "<b>kd"), out
     "<b>qd"; O = softmax(scale * Q K^T) V per batch letters <b>, scale a
     positive finite number; d must be a single block of extent 128; q and k
     block extents multiples of 128; the causal rule needs q and k of the
     same extent; bf16 data.  Scores and softmax in f32; for the P.V product
     P (in [0, 2^8]: the running max may lag the true one by up to 8 in
     the log2 domain) is rounded to fp16 and V is converted to fp16, so V
     values must lie within the fp16 range; fp32 accumulation.  The
     softmax denominator sums the same fp16 P values.
   EA_OP_SWIGLU, agg SUM: in = (X "tj", W1 "jk", W2 "jk"), out "tk" =
     silu(X W1) * (X W2), silu(g) = g / (1 + e^-g); bf16 data.
   Errors: EA_ERR_ARG, EA_ERR_SPEC, EA_ERR_DTYPE, EA_ERR_JOIN,
   EA_ERR_UNSUPPORTED, EA_ERR_HIP; EA_ERR_NOPLAN when the configuration was
   not planned on the current device (ea_joinagg_workspace); EA_ERR_CAPACITY
   when ws_bytes is below what the plan needs; EA_ERR_ARG for a missing or
   unaligned workspace the plan needs.
   workspace: caller-owned device memory, 256-byte aligned, of at least the
   bytes ea_joinagg_workspace reports (NULL and 0 if it reports 0); see
   "Workspace" above for its contents.  Asynchronous on `stream`: never
   allocates, never synchronizes. */
int ea_joinagg(const char* spec, int32_t join_op, int32_t agg_op, int32_t n_in,
               const ea_relation* const* in, ea_relation* out,
               const ea_params* params, void* workspace, int64_t ws_bytes, void* stream);

/* ---- join-agg without allocation ---------------------------------------
   For callers that cannot allocate device memory: code under HIP graph
   capture, tight serving loops, harnesses that forbid hipMalloc.  Runs a
   join-agg that ea_joinagg_workspace planned earlier on this device, like
   ea_joinagg, with the workspace taken from a library-internal device array
   of EA_NOALLOC_SCRATCH_BYTES (128 MiB) instead of a caller buffer.  It calls
   no hipMalloc, hipFree or allocating library routine: the array is part of
   the library's code object, and each GPU the library runs on holds its copy
   until the process ends.  The plan's counter words in it are cleared by a
   fill kernel on `stream` before the join-agg's kernels; the partials need no
   initial value.  Every call on one GPU shares that GPU's array, so calls that
   may overlap in time on one GPU (several streams or threads) race: issue
   them in one stream order.  Asynchronous on `stream`.  Errors as ea_joinagg
   (EA_ERR_NOPLAN if not planned), plus EA_ERR_CAPACITY when the plan's
   workspace exceeds EA_NOALLOC_SCRATCH_BYTES. */
#define EA_NOALLOC_SCRATCH_BYTES (128LL << 20)
int ea_joinagg_noalloc(const char* spec, int32_t join_op, int32_t agg_op, int32_t n_in,
                       const ea_relation* const* in, ea_relation* out,
                       const ea_params* params, void* stream);

/* Plan a join-agg configuration (the join of Section 3.2 step 1, resolved
   once as a compiled program would) and report the workspace its
   ea_joinagg calls need.  Arguments as ea_joinagg; relation data may be
   NULL.  The first call of a configuration on a device allocates the plan,
   runs the GPU join enumerator on `stream` and waits for it; later calls only
   look the plan up.  *ws_bytes: 0 when no workspace is needed, else at least
   EA_WS_COUNTER_BYTES.  Errors as ea_joinagg's validation, plus
   EA_ERR_UNSUPPORTED for a plan with more split keys than the counter area
   holds. */
int ea_joinagg_workspace(const char* spec, int32_t join_op, int32_t agg_op, int32_t n_in,
                         const ea_relation* const* in, const ea_relation* out,
                         const ea_params* params, int64_t* ws_bytes, void* stream);

/* ---- the join alone (Section 3.2 step 1, Section 3.3) -------------------
   Writes the plan's GPU-built tuple table into caller device buffers:
   tuples[n_tuples][1 + n_in] int32 = (output block, input blocks...),
   group_off[n_groups + 1] int64 CSR offsets of the groups (groups = all block
   combinations of the group letters: the output letters, minus the last one
   for RMSNORM and SOFTMAX).  Order: group-major, then the remaining letters'
   block coordinates in order of first appearance across the inputs.
   Causal (params->causal) drops a tuple iff its key block starts after its
   last query position.  Plans the configuration like ea_joinagg_workspace
   and synchronizes `stream`.  Errors as ea_joinagg, plus
   EA_ERR_CAPACITY when cap or gcap is too small (counts still written). */
int ea_join_tuples(const char* spec, int32_t join_op, int32_t n_in,
                   const ea_relation* const* in, const ea_relation* out,
                   const ea_params* params, int32_t* tuples, int64_t cap,
                   int64_t* group_off, int64_t gcap, int64_t* n_tuples,
                   int64_t* n_groups, void* stream);

/* ---- repartition (Section 5.3: overlay atoms, decompose, recompose) ------
   dst receives src's dense tensor under dst's partition.  Same rank, shape
   and dtype (EA_ERR_ARG otherwise); src and dst memory must not overlap.
   Bit-exact byte movement.  Asynchronous on `stream`: never allocates, never
   synchronizes.  EA_ERR_NOPLAN if ea_repartition_plan has not planned this
   pair of partitions (with this shape and dtype) on the current device. */
int ea_repartition(const ea_relation* src, ea_relation* dst, void* stream);
/* Plan a repartition: its overlay boxes (Section 5.3) in a library-owned
   device table.  Relation data may be NULL.  The first call for a pair of
   partitions allocates the table, uploads it on `stream` and waits; later
   calls only look it up.  Errors: EA_ERR_ARG (rank, shape or dtype differ),
   EA_ERR_UNSUPPORTED, EA_ERR_HIP. */
int ea_repartition_plan(const ea_relation* src, const ea_relation* dst, void* stream);
/* ea_repartition with an output store policy (EA_STORE_CACHED or
   EA_STORE_STREAM; other values: EA_ERR_ARG).  ea_repartition is
   ea_repartition_ex(src, dst, EA_STORE_CACHED, stream). */
int ea_repartition_ex(const ea_relation* src, ea_relation* dst, int32_t store, void* stream);

/* Overlay of two partitions of one shape (Section 5.3): per dim the sorted
   union of both split lists.  nblocks_out[rank]; splits_out must hold the
   sum over dims of (nblocks_a[d] + nblocks_b[d] + 1) entries.  Host only. */
int ea_overlay(int32_t rank, const int32_t* nblocks_a, const int64_t* splits_a,
               const int32_t* nblocks_b, const int64_t* splits_b,
               int32_t* nblocks_out, int64_t* splits_out);

/* ---- logical optimization (Section 4) -----------------------------------
   Chooses a join-agg spec for every abstract operator of a computation over
   p processors, minimising the communication proxy of Section 4.3, with the
   dynamic program over output tilings of Section 4.2 (Algorithm "Logical
   optimization").  A spec decomposes each shardable letter of the operator
   into near-equal intervals whose counts multiply to p (at most the letter's
   extent each); it is given by those counts.  Cost of a spec J with input
   tilings T_k:
     repartition: + |X_k| for each input k produced by an operator whose
                  chosen output tiling differs from the tiling J needs
                  (computation inputs are materialised as J needs: 0);
     join:        + |X_k| * p / (product of the counts of input k's letters),
                  the numbers in every function specification's k-th input;
     aggregation: + (p / (product of the output letters' counts) - 1) * |Y|,
                  the extra copies of every output block.
   Operators are listed producers first.  An output consumed once makes a
   tree edge; an output consumed several times (or by none: a designated
   output) roots a tree (Section 4.5).  Trees are optimised one at a time,
   largest first: a tensor from a tree already optimised enters with its
   chosen tiling (repartition charged), one from a tree not yet optimised
   as a computation input, whose later tiling choice is charged for the
   consumers already fixed.  Within a tree the plan is optimal. Host only. */
#define EA_LOP_MAX_INPUTS 8
typedef struct ea_lop {
  const char* spec;        /* the operator's einsum, e.g. "ij,jk->ik"              */
  const int64_t* extents;  /* extent of every distinct letter of spec, in order of
                              first appearance (inputs left to right, then output) */
  const char* shardable;   /* letters that may be split; NULL: every letter      */
  int32_t input[EA_LOP_MAX_INPUTS]; /* per input of spec: the producing operator's
                              index (lower than this one's), or -1 for a
                              computation input                                   */
} ea_lop;
/* counts: n_ops x 16 int32 (the interval count of every letter of each
   operator, letters in order of first appearance; unused entries 0).
   cost: the chosen plan's total cost under the model above.
   Errors: EA_ERR_ARG (NULL pointers, p < 1, extents < 1, a bad producer
   index); EA_ERR_SPEC (bad spec, or a producer's output shape differing from
   the consumer's input); EA_ERR_UNSUPPORTED (an operator has no spec: p is no
   product of counts within its shardable extents, or more than 2^20 specs). */
int ea_logical_plan(int32_t n_ops, const ea_lop* ops, int64_t p, int32_t* counts, int64_t* cost);

/* ---- exchange programs (Section 5.2; Definition "Closure; validity") -----
   Text of an ExProg program: declarations, then (after a blank line) a body
   of actions, statements separated by ';' or new lines.
     GPUS: 0, 1, 2, 3                      (optional: else every site named)
     PARTITIONS: G1 {size 2} G2 {0, 3}     (by size, or by members)
     IN:  A @ 0 (size: 1.0 GB); B @ 1      (atoms; size defaults to 1 GB)
     OUT: A+B @ 0, 1; C @ G1               (aggregates at sites or partitions)
     A @ 0 -> 1;  A+B @ 1 -> 2 -> 3;  A+B @ G1
   An action X @ s [-> D ...] is enabled when aggregates present at s
   partition X; firing it materialises X at s and at every destination (a
   chain -> r -> d relays through r; a source list or partition fires at
   every listed site).  The closure is the least state containing IN that is
   closed under firing enabled actions; a program is valid when every action
   is enabled by its closure and every OUT requirement is in it.  Partitions
   declared by size are valid if some membership works: partitions are
   disjoint and together cover the GPUs, members of a partition declared by
   size are drawn from the GPUs no explicit partition holds, memberships
   tried in lexicographic order.  Host only. */
/* valid: 1 or 0.  why: for an invalid program, the first OUT requirement
   missing or the first action never enabled (NUL-terminated, truncated to
   why_cap).  Errors: EA_ERR_ARG (NULL text or outputs), EA_ERR_SPEC (syntax:
   unknown site, atom or partition, malformed statement). */
int ea_exprog_check(const char* text, int32_t* valid, char* why, int64_t why_cap);
/* A valid body for the declarations of `text` (its body, if any, is ignored):
   every atom of each OUT aggregate is sent from the site holding it to each
   target site, then the aggregate is formed locally there.  Writes the
   declarations plus that body to out (NUL-terminated; *len = its length
   without the NUL; EA_ERR_CAPACITY if cap is too small, *len still set). */
int ea_exprog_naive(const char* text, char* out, int64_t cap, int64_t* len);
/* Body synthesis (Section 5.4).  Memberships of partitions declared by size
   are fixed first: the naive program is costed under each, in lexicographic
   order (the first 5040), and the cheapest is kept.  From its naive body, a
   seeded simulated-annealing search applies the paper's transformations
   (multicast fission and fusion, relay introduction and elimination,
   aggregation pushdown and pullup, source substitution) and action
   deletion; each candidate must be valid under Definition "Closure;
   validity" and is costed by ea_exprog_simulate's model.  Any body in
   text is ignored.  Writes the best program found: declarations with the
   chosen memberships written out and atom sizes in bytes, then the body;
   *seconds is its simulated time (never above the naive program's for that
   membership).  Deterministic for a given seed.  Host only.  Errors:
   EA_ERR_ARG (bad arguments, no membership under which OUT can be met),
   EA_ERR_SPEC (a syntax error), EA_ERR_CAPACITY (*len and *seconds still
   set). */
int ea_exprog_synthesize(const char* text, double link_gbs, double hbm_gbs, int32_t iters, uint64_t seed, char* out,
                         int64_t cap, int64_t* len, double* seconds);
/* Preamble of the exchange program that delivers one input of an operator
   (Section 5.3).  The producer's output is tiled by prod_nblocks/prod_splits
   (per dim nblocks[d] + 1 split points); its n_prod function specifications
   each leave one unaggregated copy of output block prod_block[i] at GPU
   prod_gpu[i].  The consumer's join-agg spec needs the input tiled by
   cons_nblocks/cons_splits; its n_cons function specifications each read
   block cons_block[j].  Atoms are the cells of the overlay of the two
   tilings, numbered from 1 in row-major order.  Writes:
     GPUS: 0, ..., n_gpus - 1
     PARTITIONS: S1 {size 1} ... Sn {size 1}     (one per consumer specification)
     IN:  <copy><atom> @ <gpu>; ...              (copy X, Y, Z, W, ... by the order
                                                  of the producer specs holding it)
     OUT: <copies of atom a, joined by +> @ <the S of every spec reading a>; ...
   IN lists producer specs in order, each with its atoms; OUT lists atoms in
   order.  elem_bytes > 0 adds each atom's size.  Host only.  Errors:
   EA_ERR_ARG (bad counts or indices, n_cons != n_gpus since the size-one
   partitions must cover the GPUs, more than 26 copies of a block),
   EA_ERR_PARTITION (split lists that do not tile one shape), EA_ERR_CAPACITY
   (*len still set). */
int ea_exprog_preamble(int32_t rank, const int32_t* prod_nblocks, const int64_t* prod_splits, int32_t n_prod,
                       const int64_t* prod_block, const int32_t* prod_gpu, const int32_t* cons_nblocks,
                       const int64_t* cons_splits, int32_t n_cons, const int64_t* cons_block, int32_t n_gpus,
                       int64_t elem_bytes, char* out, int64_t cap, int64_t* len);
/* Completion time (seconds) of a valid program on a full point-to-point mesh
   (every GPU pair linked, as xGMI connects an MI355X node): an action starts
   once its aggregate's parts are present at its source; it aggregates them
   locally (reads the parts, writes the aggregate, at hbm_gbs GB/s; nothing
   when the aggregate is present whole), then sends it along each hop, one
   transfer per destination on that pair's directed link (link_gbs GB/s).
   Stages sharing a GPU's memory or a directed link share its bandwidth
   equally.  An aggregate's size is its largest atom's.  Errors: EA_ERR_ARG
   (bad arguments, or an invalid program), EA_ERR_SPEC (syntax). */
int ea_exprog_simulate(const char* text, double link_gbs, double hbm_gbs, double* seconds);

/* ---- plan cache --------------------------------------------------------- */
/* Number of cached plans (all devices). */
int64_t ea_plan_cache_size(void);
/* Free every cached plan.  Must not run while kernels of a plan are in
   flight (it synchronizes the device of each plan first). */
int ea_plan_cache_clear(void);

#ifdef __cplusplus
}
#endif

#endif /* EA_H */
