// ea_internal.h -- structures shared by libea's host code and its HIP kernels.
//
// A plan is library-owned device memory holding what a join-agg or
// repartition needs besides the relations' data and the caller's workspace:
// the enumerator description, the split points, per-operand block tables, the
// GPU-built tuple table with its CSR group offsets and the kernel's work list.
// It is immutable once built, so calls sharing it may run concurrently on
// several streams, each with its own workspace.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "ea.h"

namespace ea {

constexpr int kMaxRank = EA_MAX_RANK;
constexpr int kMaxIn = EA_MAX_INPUTS;
constexpr int kMaxOps = EA_MAX_INPUTS + 1;  // inputs, then the output
constexpr int kMaxLetters = 16;
// A join-agg workspace: arrival counters of split keys in its first
// kWsCounterBytes (zero between calls), partial results after them.
constexpr int64_t kWsCounterBytes = EA_WS_COUNTER_BYTES;

// One block of a relation: byte offset from the relation base, and its
// sub-tensor type as (lo, extent) per dim.
struct DevBlk {
  int64_t off;
  int32_t lo[kMaxRank];
  int32_t ext[kMaxRank];
};

// ---------------------------------------------------------------------------
// Join enumerator.  Candidates are the points of the letter-block space,
// ordered group letters first (row-major), then the remaining letters in
// order of first appearance; the last letter varies fastest.  A candidate
// becomes a tuple when, for every operand, a block with exactly the
// candidate's intervals on that operand's letters is found (integer key
// matching by binary search on the operand's split points) and the optional
// causal predicate holds.
// ---------------------------------------------------------------------------
// Host helpers shared by the host sources: the thread's last error message
// (fail sets it and returns code, ok clears it and returns EA_OK) and the
// einsum spec parser.
int fail(int code, const char* fmt, ...);
int ok();

struct Spec {
  int n_in = 0;
  int rank[kMaxOps] = {};
  char let[kMaxOps][kMaxRank] = {};
};
bool is_letter(char ch);
int parse_spec(const char* s, Spec* sp);
int find_dim(const Spec& sp, int op, char l);

struct EnumDesc {
  int32_t n_in;
  int32_t n_letters;
  int32_t n_group_letters;
  int32_t causal;
  int32_t cq, ck;           // letter indices of the query/key position pair (causal, sequences)
  int32_t gqa;              // > 1: grouped-query heads, letter gh over letter gg
  int32_t gh, gg;
  int32_t n_seq;            // > 0: packed sequences, ends at splits[seq_split ..]
  int32_t seq_split;
  int64_t per_group;        // candidates per group
  int64_t n_groups;
  int64_t n_cand;
  int32_t letter_nb[kMaxLetters];
  int32_t letter_split[kMaxLetters];  // offset of the letter's driving split list
  int32_t op_rank[kMaxOps];
  int32_t op_letter[kMaxOps][kMaxRank];
  int32_t op_nb[kMaxOps][kMaxRank];
  int32_t op_split[kMaxOps][kMaxRank];  // offset of the operand's own split list
};

hipError_t launch_enumerate(const EnumDesc* d_desc, const int32_t* d_splits, int32_t* d_tuples,
                            int32_t* d_goff, int32_t* d_count, hipStream_t s);

// ---------------------------------------------------------------------------
// Generic einsum join-agg: one thread per output element, the group's tuples
// and their contracted index ranges walked in canonical order.
// ---------------------------------------------------------------------------
struct GenDesc {
  int32_t n_in, join, agg, has_res;
  int32_t out_rank, dt_out, dt_res, n_contr;
  int32_t out_letter[kMaxRank];
  int32_t in_rank[kMaxIn];
  int32_t dt_in[kMaxIn];
  int32_t in_letter[kMaxIn][kMaxRank];
  int32_t contr_letter[kMaxLetters];
  int32_t contr_op[kMaxLetters];   // input whose block gives the letter's interval
  int32_t contr_dim[kMaxLetters];
};

struct GenWork {  // one workgroup: up to 256 consecutive elements of one output block
  int32_t block;
  int32_t start;
};

struct GenArgs {
  const GenDesc* desc;
  const int32_t* tuples;
  const int32_t* goff;
  const DevBlk* blk[kMaxOps];  // inputs, then output
  const char* in[kMaxIn];
  char* out;
  const char* res;
  const GenWork* work;
  int64_t n_work;
};

hipError_t launch_generic(const GenArgs& a, hipStream_t s);

// ---------------------------------------------------------------------------
// Repartition: the overlay of the source and destination partitions cuts the
// tensor into boxes, each inside exactly one source block and one destination
// block; a task copies a range of a box's rows (rows run along the last dim).
// ---------------------------------------------------------------------------
struct RepTask {
  int64_t src_off, dst_off;         // bytes from the bases to the box origin
  int64_t src_stride[kMaxRank - 1]; // bytes per step of each outer dim
  int64_t dst_stride[kMaxRank - 1];
  int32_t outer_ext[kMaxRank - 1];  // extents of the outer dims
  int32_t n_outer;
  int32_t row_bytes;
  int32_t vec;                      // bytes per vector access: 16, 8, 4, 2 or 1
  int32_t begin, end;               // byte range of the box (rows x row_bytes) copied
  int32_t row_shift;                // log2(row_bytes) when a power of two, else -1
  int32_t pad;
};

// A task copies kRepTaskBytes of one box (one pass of 256 lanes x 4 x 16
// bytes) in relations of at least kRepLargeBytes, else kRepTaskBytesSmall (256
// lanes x 2 x 16 bytes): where the whole copy takes a few microseconds,
// smaller tasks put more workgroups to work at once.
constexpr int kRepTaskBytes = 16384;
constexpr int kRepTaskBytesSmall = 8192;
constexpr int64_t kRepLargeBytes = int64_t(64) << 20;
hipError_t launch_repartition(const RepTask* d_tasks, int64_t n_tasks, const char* src, char* dst, bool stream_out,
                              bool small_tasks, hipStream_t s);

// ---------------------------------------------------------------------------
// Block GEMM on the matrix cores: out = sum over the group's tuples of
// A_blk * B_blk (+ residual), bf16/f16 inputs, fp32 accumulation.
// ---------------------------------------------------------------------------
constexpr int kGemmTM = 256;          // output tile rows of one workgroup
constexpr int kGemmTN = 256;          // output tile columns (128 for SwiGLU)
constexpr int kGemmTNSwiglu = 128;
constexpr int kGemmMaxTuples = 128;   // tuples per unit on the direct-to-LDS kernel

struct GemmTile {      // one workgroup: a tile of one output block and a run of its tuples
  int32_t block;       // output block == group index
  int32_t m0, n0;
  int32_t part;        // tuples [part*n/n_parts, (part+1)*n/n_parts) of the group's n
  int32_t n_parts;
  int32_t slot;        // partial-sum slot (split tiles only)
  int32_t first_slot;  // first slot of the tile's parts
  int32_t counter;     // arrival counter of the tile (split tiles only)
};

// Direct-load kernel: a workgroup's unit is up to kGemmMaxSegs segments, each a
// run of 32-deep K steps of one output tile.  Balanced units take equal runs of
// the tiles' K steps laid end to end, so a unit may finish one tile and start
// the next; a tile cut into several segments is merged by its last arriver.
struct GemmSeg {
  int32_t block, m0, n0;  // output tile
  int32_t s0, s1;         // K steps [s0, s1) of the tile's walk over its group's tuples
  int32_t part, n_parts;  // place among the tile's segments (ascending s0); n_parts 1: not split
  int32_t first_slot;     // split tile: part i's partial sums go to workspace slot first_slot + i
  int32_t counter;        // split tile: its arrival counter
  // resolved from the GPU join at plan time (launch_gemm_prep): the group's
  // first tuple and tuple count, the tuple holding step s0 and the steps of
  // it before s0, and the segment's step count (s1 clamped to the group's)
  int32_t gb, nt, t0, skip, n_steps;
  int32_t pad[2];
};
static_assert(sizeof(GemmSeg) == 64, "GemmSeg layout");

// Operand blocks of one tuple of the direct-load kernel, in tuple-table
// order (written at plan time from the tuple table and the block records).
struct GemmTupleMeta {
  int64_t aoff, boff, b2off;  // block byte offsets in A, B and (SwiGLU) B2
  int32_t am, ak;             // A block extents
  int32_t b0, b1, b20, b21;   // B and B2 block extents
  int32_t pad[4];
};
static_assert(sizeof(GemmTupleMeta) == 64, "GemmTupleMeta layout");
constexpr int kGemmMaxSegs = 2;
struct GemmUnit {
  GemmSeg seg[kGemmMaxSegs];
  int32_t n_seg, pad[3];
};

struct GemmArgs {
  const int32_t* tuples;
  const int32_t* goff;
  const DevBlk* blk_a;
  const DevBlk* blk_b;
  const DevBlk* blk_b2;  // second right operand (SwiGLU), else null
  const DevBlk* blk_c;
  const char* a;
  const char* b;
  const char* b2;
  char* c;
  const char* res;       // residual relation data (same layout as c) or null
  const GemmTile* tiles;  // register-staged kernel: one tile and run of tuples per workgroup
  int32_t n_tiles;
  const GemmUnit* units;  // direct-load kernel: one unit per workgroup
  int32_t n_units;
  int32_t tuple_stride;  // 1 + n_in
  int32_t b_kmajor;      // 1: B blocks are [n][k] ("ab,cb->ac"); 0: [k][n]
  int32_t dt_in;         // EA_BF16 or EA_F16
  int32_t dt_out;        // EA_F32, EA_BF16 or EA_F16
  int32_t dt_res;
  int32_t swiglu;        // 1: out = silu(A B) * (A B2)
  int32_t direct;        // 1: direct-to-LDS kernel (contracted block extents multiples of 32)
  int32_t tile_n;        // output tile columns per right operand: 256, or 128 (SwiGLU, or a narrow plan)
  GemmTupleMeta* meta;   // direct-load kernel: per-tuple operand blocks (plan time)
  const int32_t* count;  // number of tuples of the join (plan time)
  float* partials;       // [slots][256 x 256] fp32 partial sums of split tiles
  int32_t* counters;     // one per split tile; zero between calls
};

hipError_t launch_gemm(const GemmArgs& a, hipStream_t s);
// Plan time, after the join: fills a.meta (tuple_cap entries) and the
// join-derived fields of every segment of a.units (direct-load plans).
hipError_t launch_gemm_prep(const GemmArgs& a, GemmUnit* units, int64_t tuple_cap, hipStream_t s);

// ---------------------------------------------------------------------------
// fp32 block product "ab,bc->ac" / "ab,cb->ac" on the vector ALUs: a workgroup
// owns a kGemm32Tile-square tile of one output block and sums its key's tuples.
// ---------------------------------------------------------------------------
constexpr int kGemm32Tile = 32;
struct Gemm32Work {
  int32_t block, m0, n0, pad;
};

struct Gemm32Args {
  const int32_t* tuples;
  const int32_t* goff;
  const DevBlk* blk_a;
  const DevBlk* blk_b;
  const DevBlk* blk_c;
  const char* a;
  const char* b;
  char* c;
  const Gemm32Work* work;
  int64_t n_work;
  int32_t tuple_stride;
  int32_t b_kmajor;  // 1: B blocks are [n][k] ("ab,cb->ac")
  int32_t dt_out;    // EA_F32, EA_BF16 or EA_F16
};

hipError_t launch_gemm32(const Gemm32Args& a, hipStream_t s);

// ---------------------------------------------------------------------------
// Row reductions.  A row is the concatenation of its segments, one per tuple
// of its group (RMSNorm: column blocks of x with the matching w blocks;
// softmax: key blocks).
// ---------------------------------------------------------------------------
// One workgroup's rows: up to four consecutive rows of one group.  The
// remaining fields serve the affine layout (see RowArgs::affine): the query
// block's start and extent along the causal letter, and the byte offsets of
// the task's first row in the group's first x and y blocks.
struct RowTask {
  int32_t g, row0, nrows, qlo;
  int32_t qext, pad;
  int64_t xrow, yrow;
};

struct RowArgs {
  const int32_t* tuples;
  const int32_t* goff;
  const DevBlk* blk_x;
  const DevBlk* blk_w;   // RMSNorm weight blocks, or null
  const DevBlk* blk_y;
  const char* x;
  const char* w;
  char* y;
  const RowTask* tasks;  // one per workgroup
  int32_t n_rowtasks;
  int32_t tuple_stride;
  int32_t rank;          // rank of x / y
  int32_t dt_x, dt_w, dt_y;
  int32_t causal;        // softmax: mask keys beyond the row's query position
  int32_t row_len;       // full extent of the normalised letter
  int32_t vec;           // 1: register path (see rows_vec_ok)
  int32_t seg_chunks;    // register path: 16-byte chunks of every segment but the
                         // last (which has at most as many), or 0 if uneven
  float seg_inv;         // 1 / seg_chunks (fp32), or 0
  float eps;
  // Affine layout (set on the host when it holds): every segment has seg_len
  // elements, x, y and w have the same partition of the normalised letter,
  // and segment s of a row sits at a fixed byte stride from segment 0 (xs,
  // ys, ws; w's segment 0 at wbase).  Every address then follows from the
  // task record, with no tuple or block-table loads before the row loads.
  int32_t affine;
  int32_t stream_out;    // non-temporal output stores (EA_STORE_STREAM)
  int32_t seg_len, nseg;
  int64_t xs, ys, ws, wbase;
};

bool rows_vec_ok(int64_t row_len, int64_t max_segments, bool seg_aligned, int es);

hipError_t launch_rmsnorm(const RowArgs& a, hipStream_t s);
hipError_t launch_softmax(const RowArgs& a, hipStream_t s);

// ---------------------------------------------------------------------------
// Causal attention with key-split online-softmax aggregation.
// A unit is (group, query tile of 128 rows, a run of the group's tuples).
// Units of one (group, tile) that split its tuples write partial (m, l, O)
// to the caller's workspace; the last unit to finish merges them in tuple
// order.
// ---------------------------------------------------------------------------
struct AttnUnit {
  int32_t group;
  int32_t q0;          // first query row inside the q block
  int32_t part;        // this unit takes tuples [part*n/n_parts, (part+1)*n/n_parts)
  int32_t n_parts;     //   of its group's n tuples
  int32_t slot;        // partial slot of this unit, -1 when the unit is alone
  int32_t first_slot;  // first slot of the (group, tile), for the merge
  int32_t counter;     // arrival counter index of the (group, tile)
  int32_t weight;      // expected tuple count (host-side ordering only)
};

constexpr int kRowsPerTask = 4;  // RMSNorm/softmax row tasks: rows per workgroup, one per wavefront
constexpr int kAttnMaxUnitTuples = 64;  // key blocks per attention work unit (LDS table size)

// Per-unit block metadata, resolved once per plan from the GPU-built tuple
// table (attention prep kernel), so that the attention kernel reaches its
// first loads without the chain unit -> group offsets -> tuples -> blocks.
struct AttnKv {
  int64_t koff, voff;  // byte offsets of the K and V blocks
  int32_t klo, kext;   // key interval of the block
};
constexpr int kAttnChunkKeys = 64;  // keys the attention kernel stages per chunk
constexpr int kAttnTileRows = 128;  // query rows of an attention work unit
struct AttnUnitMeta {
  int64_t qoff, ooff;  // byte offsets of the unit's Q and O blocks
  int32_t q_lo, nt;    // query position of the Q block's first row; the unit's tuples
  int32_t nc;          // kAttnChunkKeys-key chunks of the unit's walk (causal cut applied)
  int32_t n_plain;     // leading chunks of the walk that the causal rule masks for no query of the tile
  AttnKv kv[kAttnMaxUnitTuples];
};

struct AttnArgs {
  const int32_t* tuples;
  const int32_t* goff;
  const DevBlk* blk_q;
  const DevBlk* blk_k;
  const DevBlk* blk_v;
  const DevBlk* blk_o;
  const char* q;
  const char* k;
  const char* v;
  char* o;
  const AttnUnit* units;
  int32_t n_units;
  int32_t causal;
  int32_t q_dim, k_dim;  // dim index of q (in Q/O) and k (in K/V)
  float scale;
  float* part_o;         // [slots][128 rows][128] fp32
  float* part_ml;        // [slots][128 rows][2]
  int32_t* counters;     // one per split (group, tile); zero between calls
  int32_t dt_o;
  AttnUnitMeta* meta;    // one per unit (written by the prep kernel at plan time)
  int32_t* overflow;     // prep kernel: set to 1 if a unit exceeds kAttnMaxUnitTuples
};

hipError_t launch_attention(const AttnArgs& a, hipStream_t s);
// Plan time: fill a.meta from the tuple table (a's data pointers unused).
hipError_t launch_attention_prep(const AttnArgs& a, hipStream_t s);

}  // namespace ea
