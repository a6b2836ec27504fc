// ea_attn.hip -- causal attention join-agg with key-blocked online-softmax
// aggregation.
//
// Section 3.3, Example "Flash attention" names the operator; here the tuples
// of an output key (batch letters, query block) are its key/value blocks, the
// per-tuple operator computes a partial (m, l, O) for those keys, and the
// aggregation is the online-softmax combine
//   m = max(m1, m2), l = l1 2^(m1-m) + l2 2^(m2-m), O = O1 2^(m1-m) + O2 2^(m2-m)
// (scores are kept in the log2 domain), associative and commutative, applied
// in ascending key-block order.
//
// Work unit = (group, 128-row query tile, a run of the group's tuples).  A
// workgroup is 4 waves x 32 query rows, and two workgroups share a CU: they
// meet at no common barrier, so one's softmax VALU work runs beside the
// other's MFMAs.  Every wave computes each 64-key chunk of the walk while
// the workgroup's loads of the next chunk land in the other of two 32 KiB
// buffers; each wave issues its share of them one per score step, so that a
// wave held by the load path waits under its own running MFMAs.  Per
// 64-key chunk:
//   * K and V chunks [key][d] (bf16, 256-byte rows) go straight from global
//     memory into LDS (global_load_lds_dwordx4), their 16-byte chunks
//     XOR-swizzled per key row so that the fragment reads below spread over
//     all banks;
//   * S^T = K Q^T on bf16 MFMA 32x32x16 (Q^T from registers), so each lane
//     holds the scores of one query: the row max and sum need one exchange
//     between lanes l and l^32;
//   * while those MFMAs run, each wave converts the V pieces it loaded to
//     fp16 in place (exact for values in fp16's normal range), and the
//     workgroup meets;
//   * the scale (log2 domain) is one FMA ahead of exp2; the causal mask is
//     applied only on chunks that reach past a query of the wave;
//   * P = 2^(S - m), in [0, 2^8] (m lags the true max by at most 8), is
//     rounded to fp16; the row sum adds those fp16 values (v_dot2_f32_f16)
//     and O^T += V^T P^T runs on fp16 MFMA 32x32x16; the V^T
//     operand (8 keys of one d per lane) comes from two transposing LDS reads
//     (ds_read_b64_tr_b16) of the [key][d] chunk, with the MFMA's k order
//     matched to the accumulator layout of S^T.
// A group whose tuples are split across units writes partial (m, l, O) to the
// workspace; the last unit to arrive (device-scope counter, no waiting)
// merges the partials in a fixed order and stores the output block rows.
#include "ea_device.h"

namespace ea {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;       // 4 waves x 32 query rows
constexpr int D = 128;              // head dim
constexpr int KC = kAttnChunkKeys;  // keys per staged chunk (64)
constexpr int KT = KC / 32;         // 32-key MFMA tiles per chunk
constexpr int LPW = KC / 16;        // direct loads (4 key rows each) per wave per chunk, for K and for V each
constexpr int BUF = 2 * KC * D;     // LDS elements per chunk buffer: K chunk, then V chunk
constexpr int NBUF = 2;             // one chunk computed while the next loads

// Per-tuple K/V metadata of a unit, staged in LDS once so that the chunk walk
// never waits on a chain of global table loads.
struct KvMeta {
  int64_t koff, voff;  // byte offsets of the K and V blocks
  int32_t klo, kext;   // key interval of the block
};
constexpr float kLog2e = 1.4426950408889634f;
template <bool B>
struct Bool { static constexpr bool value = B; };
constexpr float kLazyMax = 8.0f;  // log2 of the largest P the lazy running max allows

typedef short s16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x16_t mfma_bf16(const uint4& a, const uint4& b, const f32x16_t& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                  c, 0, 0, 0);
}

typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));


// acc + x.lo + x.hi for a packed fp16 pair x (v_dot2_f32_f16 against 1, 1)
__device__ __forceinline__ float sum_f16x2(uint32_t x, float acc) {
  const f16x2_t one = {(_Float16)1.0f, (_Float16)1.0f};
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2_t, x), one, acc, false);
}

// two floats -> packed fp16 pair, round to nearest even (v_cvt_pk_f16_f32)
__device__ __forceinline__ uint32_t pack_f16(float x0, float x1) {
  const f16x2_t h = {(_Float16)x0, (_Float16)x1};
  return __builtin_bit_cast(uint32_t, h);
}

// packed bf16 pair -> packed fp16 pair (exact for values in the fp16 normal range)
__device__ __forceinline__ uint32_t bf16x2_to_f16x2(uint32_t w) {
  return pack_f16(__uint_as_float(w << 16), __uint_as_float(w & 0xffff0000u));
}

// K chunk: logical 16-byte chunk c of key row r at physical chunk c ^ (r & 15)
// (the 16 rows read by 16 lanes hit 16 distinct chunks).
__device__ __forceinline__ int swz_krow(int r) { return r & 15; }
// V chunk: the 4 key rows of one transposing read take disjoint chunk sets
// (for 16-lane groups over 32 banks and 32-lane groups over 64 banks).
__device__ __forceinline__ int swz_vrow(int r) { return (2 * (r & 3)) ^ (8 * (r & 1)); }

// One direct global->LDS load: each lane fetches 16 bytes at base + voff
// (base wave-uniform, in scalar registers; voff a 32-bit per-lane offset) and
// the wave's 64 pieces land contiguously at LDS byte address lds_addr.
// Issued through inline asm so that the compiler does not track the LDS
// write; the kernel waits for it explicitly (vmcnt 0, then a barrier).
// Nothing else in this kernel reads M0, so the warning for the reserved
// register is silenced.
__device__ __forceinline__ void dl_load16(const char* base, uint32_t voff, uint32_t lds_addr) {
  const uint32_t lds = __builtin_amdgcn_readfirstlane(lds_addr);
  // readfirstlane yields an int: widen through uint32_t, never by sign extension
  const uint64_t b = (uint64_t)(uintptr_t)base;
  const uint32_t b_lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b);
  const uint32_t b_hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
  const uint64_t sbase = (uint64_t)b_lo | ((uint64_t)b_hi << 32);
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
#pragma clang diagnostic pop
}

__device__ __forceinline__ s16x4 tr_read(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)p);
}
// the PV MFMA's A operand from two transposing reads, concatenated as one
// vector (so that the reads can land in the operand's registers directly)
typedef short s16x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ f32x16_t mfma_f16_tr(const s16x4& lo, const s16x4& hi, const uint4& b, const f32x16_t& c) {
  const s16x8 a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b), c, 0,
                                                 0, 0);
}

// 2^x on the transcendental unit; arguments here are at most kLazyMax, and
// results below the normal range contribute nothing next to the at least 1
// of the row's largest term.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__global__ __launch_bounds__(kThreads, 2) void attn_kernel(const AttnArgs p) {
  __shared__ __attribute__((aligned(1024))) uint16_t sKV[NBUF * BUF];  // chunk buffers: K, then V
  __shared__ KvMeta s_tm[kAttnMaxUnitTuples];
  __shared__ int s_last;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wq = wid;  // wave: query rows 32 wq .. 32 wq + 31 of the tile
  const int g = lane >> 5, lq = lane & 31;
  const AttnUnit u = p.units[blockIdx.x];
  // the unit's blocks, resolved at plan time from the tuple table
  const AttnUnitMeta& um = p.meta[blockIdx.x];
  const int nt = ld_uniform(&um.nt);
  const int nc = ld_uniform(&um.nc);  // chunks of the walk, up to the first past the tile's last query
  // leading chunks that no query of the tile masks, rounded down to even so
  // that the rest of the walk starts on buffer 0
  const int n_plain = ld_uniform(&um.n_plain) & ~1;
  const int q_lo = ld_uniform(&um.q_lo);
  const int64_t qoff = ld_uniform(&um.qoff), ooff = ld_uniform(&um.ooff);
  // the first tuple's K/V record, read with the fields above (one round trip
  // of scalar loads, not two): kv[0] is part of every unit's record, and is
  // used only when the walk has a chunk
  const int64_t ko0 = ld_uniform(&um.kv[0].koff), vo0 = ld_uniform(&um.kv[0].voff);
  const int klo0 = ld_uniform(&um.kv[0].klo), kext0 = ld_uniform(&um.kv[0].kext);
  // an empty statement that takes the four values keeps the compiler from
  // sinking their loads into the branch below, behind a wait of their own
  asm volatile("" ::"s"(ko0), "s"(vo0), "s"(klo0), "s"(kext0));
  const int row = u.q0 + wq * 32 + lq;  // this lane's query row inside the block
  const int qpos = q_lo + row;          // its position
  const int qpos_wave_min = q_lo + u.q0 + wq * 32;
  const int qpos_wave_max = qpos_wave_min + 31;
  const float sc = p.scale * kLog2e;
  const bool causal = p.causal != 0;
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint16_t*)sKV;

  // walk of the chunks in load order; chunk j goes to buffer j % NBUF
  int it_t = 0, it_c = 0;  // tuple (index into s_tm) and offset of the next chunk to load
  int key0_buf[NBUF];  // first key of the chunk held in each buffer (constant indices only)
#pragma unroll
  for (int b = 0; b < NBUF; ++b) key0_buf[b] = 0;

  // Issue the K or the V loads of one chunk into buffer b (a compile-time
  // constant): all 4 waves take part, LPW loads of 4 key rows each per wave.
  auto issue_k = [&](int b, const char* kbase) {
    const uint32_t ldsK = lds0 + b * BUF * 2;
#pragma unroll
    for (int q = 0; q < LPW; ++q) {
      const int inst = wid * LPW + q;
      const int r = inst * 4 + (lane >> 4);  // key row of this lane's piece
      dl_load16(kbase, (uint32_t)((r * D + 8 * ((lane & 15) ^ swz_krow(r))) * 2), ldsK + inst * 1024);
    }
  };
  auto issue_v = [&](int b, const char* vbase) {
    const uint32_t ldsV = lds0 + b * BUF * 2 + KC * D * 2;
#pragma unroll
    for (int q = 0; q < LPW; ++q) {
      const int inst = wid * LPW + q;
      const int r = inst * 4 + (lane >> 4);
      dl_load16(vbase, (uint32_t)((r * D + 8 * ((lane & 15) ^ swz_vrow(r))) * 2), ldsV + inst * 1024);
    }
  };
  // one of a chunk's 2 LPW loads of this wave: q < LPW a K piece, else a V piece
  auto issue_piece = [&](int b, int q, const char* kbase, const char* vbase) {
    const int qq = q % LPW, inst = wid * LPW + qq;
    const int r = inst * 4 + (lane >> 4);
    if (q < LPW)
      dl_load16(kbase, (uint32_t)((r * D + 8 * ((lane & 15) ^ swz_krow(r))) * 2), lds0 + b * BUF * 2 + inst * 1024);
    else
      dl_load16(vbase, (uint32_t)((r * D + 8 * ((lane & 15) ^ swz_vrow(r))) * 2),
                lds0 + b * BUF * 2 + KC * D * 2 + inst * 1024);
  };
  auto advance = [&](int kext) {
    it_c += KC;
    if (it_c >= kext) {
      ++it_t;
      it_c = 0;
    }
  };

  // The first chunk goes out first, its addresses taken from the record by
  // scalar loads (before the metadata table reaches LDS, and before Q).
  if (nc > 0) {
    key0_buf[0] = klo0;
    issue_k(0, p.k + ko0);
    issue_v(0, p.v + vo0);
    advance(kext0);
  }

  // the unit's tuples' K/V metadata (nt <= kAttnMaxUnitTuples: host guarantee)
  AttnKv kv{};
  if (tid < nt) kv = um.kv[tid];

  // Q^T operand: lane holds Q[row][16 s + 8 g .. + 7] for s = 0..7
  uint4 qreg[8];
  {
    const char* qrow = p.q + qoff + (int64_t)row * D * 2;
#pragma unroll
    for (int s = 0; s < 8; ++s) qreg[s] = *reinterpret_cast<const uint4*>(qrow + (16 * s + 8 * g) * 2);
  }

  f32x16_t acc_o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc_o[i] = f32x16_t{};
  float m = -INFINITY, l = 0.0f;  // running max (log2 domain, scaled) and sum

  // metadata into LDS; it is read after the prologue barrier below
  if (tid < nt) {
    KvMeta mt;
    mt.koff = kv.koff;
    mt.voff = kv.voff;
    mt.klo = kv.klo;
    mt.kext = kv.kext;
    s_tm[tid] = mt;
  }

  // The next chunk of the walk (metadata from LDS) for buffer b: its first
  // key, and its K and V block addresses.
  auto next_chunk = [&](int b, const char*& kbase, const char*& vbase) {
    const KvMeta& mt = s_tm[it_t];
    key0_buf[b] = mt.klo + it_c;
    kbase = p.k + mt.koff + (int64_t)it_c * D * 2;
    vbase = p.v + mt.voff + (int64_t)it_c * D * 2;
    advance(mt.kext);
  };
  // after this wave's loads have landed: its V pieces of buffer b to fp16
  auto convert_v = [&](int b) {
    uint16_t* sVb = sKV + b * BUF + KC * D;
#pragma unroll
    for (int q = 0; q < LPW; ++q) {
      uint4* piece = reinterpret_cast<uint4*>(sVb + (wid * LPW + q) * 512 + lane * 8);
      const uint4 w = *piece;
      *piece = make_uint4(bf16x2_to_f16x2(w.x), bf16x2_to_f16x2(w.y), bf16x2_to_f16x2(w.z), bf16x2_to_f16x2(w.w));
    }
  };

  // compute the 64-key chunk held in buffer b: S^T = K Q^T, an online
  // softmax step, O^T += V^T P^T.  DIAG: some key of the chunk is past some
  // query of the wave, so the causal mask is applied (a separate
  // instantiation: the other chunks carry no mask arithmetic at all).
  auto compute_chunk_impl = [&](int b, auto diag_tag, auto&& load) {
    constexpr bool DIAG = decltype(diag_tag)::value;
    const uint16_t* sK = sKV + b * BUF;
    const uint16_t* sV = sK + KC * D;
    const int key0 = key0_buf[b];
    f32x16_t acc_s[KT];
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) acc_s[kt] = f32x16_t{};
    // wave priority up while this wave's MFMAs issue: the SIMD's other wave
    // (the other workgroup's) fills the gaps with its VALU work
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      uint4 a[KT];
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) {
        const int r = 32 * kt + lq;
        a[kt] = *reinterpret_cast<const uint4*>(sK + r * D + 8 * ((2 * s + g) ^ swz_krow(r)));
      }
      load(s);  // one of the next chunk's loads per step, behind running MFMAs
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) acc_s[kt] = mfma_bf16(a[kt], qreg[s], acc_s[kt]);
    }
    __builtin_amdgcn_s_setprio(0);
    // online softmax in the log2 domain; the scale is one FMA ahead of exp2
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float sv = acc_s[kt][r];
        if (DIAG) {
          const int kpos = key0 + 32 * kt + 8 * (r >> 2) + 4 * g + (r & 3);
          sv = kpos > qpos ? -INFINITY : sv;
          acc_s[kt][r] = sv;
        }
        mx = fmaxf(mx, sv);
      }
    mx = fmaxf(mx, other32(mx));  // the lane-pair exchange, no LDS round trip
    // The running max moves only when a score passes it by more than
    // kLazyMax (log2 domain).  O / l is the same for any m the two share, P
    // stays at most 2^kLazyMax (exact range and precision in fp16), and the
    // rescale of O below is skipped on most chunks.
    const float cand = mx * sc;
    const float m_new = cand > m + kLazyMax ? cand : m;
    const float m_use = m_new == -INFINITY ? 0.0f : m_new;
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc_s[kt][r] = fast_exp2(fmaf(acc_s[kt][r], sc, -m_use));
    if (__any(m_new != m)) {  // a running max moved: rescale (else alpha is 1 on every lane)
      const float alpha = fast_exp2(m - m_use);
      l *= alpha;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc_o[dt][r] *= alpha;
    }
    m = m_new;
    // MFMA k index 8 g + e maps to key 32 kt + 16 h + 4 g + e (e < 4) or
    // 32 kt + 16 h + 8 + 4 g + (e - 4); P in fp16 (RNE), V in fp16
    const int gq = lane >> 4, li = lane & 15;
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint4 ph = make_uint4(pack_f16(acc_s[kt][8 * h], acc_s[kt][8 * h + 1]),
                                    pack_f16(acc_s[kt][8 * h + 2], acc_s[kt][8 * h + 3]),
                                    pack_f16(acc_s[kt][8 * h + 4], acc_s[kt][8 * h + 5]),
                                    pack_f16(acc_s[kt][8 * h + 6], acc_s[kt][8 * h + 7]));
        // the row sum takes the same fp16 P as the PV product, two terms per
        // v_dot2_f32_f16 (this lane's half of the row: the pair's halves
        // are added once after the walk, as both share every running max)
        l = sum_f16x2(ph.x, l);
        l = sum_f16x2(ph.y, l);
        l = sum_f16x2(ph.z, l);
        l = sum_f16x2(ph.w, l);
        const int k0 = 32 * kt + 16 * h + 4 * (gq >> 1) + (li >> 2);  // key row of this lane's first read
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) {
          const int d = 32 * dt + 16 * (gq & 1) + 4 * (li & 3);
          const s16x4 v0 = tr_read(sV + k0 * D + 8 * ((d >> 3) ^ swz_vrow(k0)) + (d & 4));
          const s16x4 v1 = tr_read(sV + (k0 + 8) * D + 8 * ((d >> 3) ^ swz_vrow(k0 + 8)) + (d & 4));
          acc_o[dt] = mfma_f16_tr(v0, v1, ph, acc_o[dt]);
        }
      }
    __builtin_amdgcn_s_setprio(0);
  };
  auto compute_chunk = [&](int b, auto&& load) {
    const int key0 = key0_buf[b];
    if (causal && key0 > qpos_wave_max) {  // the whole wave is masked in this chunk
#pragma unroll
      for (int q = 0; q < 2 * LPW; ++q) load(q);
    } else if (causal && key0 + KC - 1 > qpos_wave_min) {
      compute_chunk_impl(b, Bool<true>{}, load);
    } else {
      compute_chunk_impl(b, Bool<false>{}, load);
    }
  };

  // The walk: chunk j is computed from buffer j % 2 while every wave issues
  // its loads of chunk j + 1 into the other buffer (which all waves finished
  // with before the previous barrier); then each wave waits for its own
  // loads, turns the V pieces it loaded to fp16 in place, and the workgroup
  // meets at the barrier (one per chunk).
  // The loop runs two chunks per iteration so that every buffer index is a
  // compile-time constant.  (Earlier designs measured: eight
  // waves in two groups computing alternate chunks of one tile, with four
  // buffers, spent most of each phase with both waves of a SIMD in the same
  // stage -- MFMA, then VALU -- and were slower; so were 32-key chunks with
  // three phases of lookahead, and V transposed to [d][key] once per chunk.)
  // s_waitcnt vmcnt(0) (gfx9 encoding; expcnt and lgkmcnt at their maxima)
  auto wait_loads = [&]() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));
    asm volatile("" ::: "memory");
  };
  wait_loads();
  if (nc > 0) convert_v(0);
  __syncthreads();
  // Chunks that no query of the tile masks run in a loop of their own with
  // the unmasked chunk code alone: with one path through the loop, O keeps
  // its registers from one chunk to the next (where the masked, unmasked
  // and fully masked paths meet, the compiler moves all of O between
  // register sets after each chunk's last MFMA).
  for (int j0 = 0; j0 < n_plain; j0 += NBUF) {
#pragma unroll
    for (int e = 0; e < NBUF; ++e) {
      const int j = j0 + e;  // < n_plain (even)
      const char *kb = nullptr, *vb = nullptr;
      const bool more = j + 1 < nc;
      if (more) next_chunk(1 - e, kb, vb);
      compute_chunk_impl(e, Bool<false>{}, [&](int q) {
        if (more) issue_piece(1 - e, q, kb, vb);
      });
      if (more) {
        wait_loads();
        convert_v(1 - e);
      }
      __syncthreads();
    }
  }
  for (int j0 = n_plain; j0 < nc; j0 += NBUF) {
#pragma unroll
    for (int e = 0; e < NBUF; ++e) {
      const int j = j0 + e;
      if (j < nc) {
        // the next chunk's loads go out one per score step, so that a wave
        // held by the load path waits under its own running MFMAs; after
        // its PV MFMAs are issued, each wave waits for its own loads and
        // turns its V pieces of the next chunk to fp16 while they run, and
        // the workgroup meets once per chunk
        const char *kb = nullptr, *vb = nullptr;
        const bool more = j + 1 < nc;
        if (more) next_chunk(1 - e, kb, vb);
        compute_chunk(e, [&](int q) {
          if (more) issue_piece(1 - e, q, kb, vb);
        });
        if (more) {
          wait_loads();
          convert_v(1 - e);
        }
        __syncthreads();
      }
    }
  }

  l += other32(l);  // the row's two halves (lanes l and l^32)

  // ---- split group: write this unit's partial (m, l, O), the last unit of
  // the (group, tile) merges in registers.  Partials go through the plan's
  // scratch with the sc1 cache policy (coherent between the XCDs' L2s): O as
  // lane-contiguous 16-byte pieces (every store writes whole lines), (m, l)
  // as one 8-byte pair per query row.
  if (u.slot >= 0) {
    constexpr int kCoherent = 16;  // sc1
    auto o_rsrc = [&](int slot) {
      return __builtin_amdgcn_make_buffer_rsrc(p.part_o + (int64_t)slot * 128 * D, 0, 0x7fffffff, 0x00020000);
    };
    auto ml_rsrc = [&](int slot) {
      return __builtin_amdgcn_make_buffer_rsrc(p.part_ml + (int64_t)slot * 128 * 2, 0, 0x7fffffff, 0x00020000);
    };
    auto o_piece = [&](int q) { return (uint32_t)(((wq * 16 + q) * 64 + lane) * 16); };
    const uint32_t ml_off = (uint32_t)((wq * 32 + lq) * 8);
    {
      const auto ro = o_rsrc(u.slot);
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const f32x16_t& c = acc_o[q / 4];
        const int r0 = 4 * (q % 4);
        const u32x4_t v = {__float_as_uint(c[r0]), __float_as_uint(c[r0 + 1]), __float_as_uint(c[r0 + 2]),
                           __float_as_uint(c[r0 + 3])};
        __builtin_amdgcn_raw_buffer_store_b128(v, ro, o_piece(q), 0, kCoherent);
      }
      if (g == 0) {
        const u32x2_t ml = {__float_as_uint(m), __float_as_uint(l)};
        __builtin_amdgcn_raw_buffer_store_b64(ml, ml_rsrc(u.slot), ml_off, 0, kCoherent);
      }
    }
    drain_vmem();
    __syncthreads();
    if (tid == 0) s_last = arrive_agent(p.counters + u.counter) == u.n_parts - 1;
    __syncthreads();
    if (!s_last) return;
    if (tid == 0) reset_agent(p.counters + u.counter);  // ready for the next call (stream-ordered)
    auto load_ml = [&](int slot) {
      const u32x2_t v = __builtin_amdgcn_raw_buffer_load_b64(ml_rsrc(slot), ml_off, 0, kCoherent);
      return make_float2(__uint_as_float(v.x), __uint_as_float(v.y));
    };
    // one part's partial, its 16 O pieces and its (m, l), in one batch of
    // loads
    auto load_part = [&](int slot, u32x4_t (&o)[16], float2& ml) {
      ml = load_ml(slot);
      const auto ro = o_rsrc(slot);
#pragma unroll
      for (int t = 0; t < 16; ++t) o[t] = __builtin_amdgcn_raw_buffer_load_b128(ro, o_piece(t), 0, kCoherent);
    };
    // acc_o = a_own * acc_o + w * O_part; both products rounded before the
    // add (no fused multiply-add)
    auto add_part = [&](const u32x4_t (&o)[16], float a_own, float w) {
#pragma unroll
      for (int t = 0; t < 16; ++t) {
#pragma clang fp contract(off)
        f32x16_t& c = acc_o[t / 4];
        const int r0 = 4 * (t % 4);
        c[r0] = c[r0] * a_own + __uint_as_float(o[t].x) * w;
        c[r0 + 1] = c[r0 + 1] * a_own + __uint_as_float(o[t].y) * w;
        c[r0 + 2] = c[r0 + 2] * a_own + __uint_as_float(o[t].z) * w;
        c[r0 + 3] = c[r0 + 3] * a_own + __uint_as_float(o[t].w) * w;
      }
    };
    const int np = u.n_parts;
    if (np == 2) {
      // own + other: every term is formed the same way whichever part holds
      // it, and a + b == b + a exactly, so the bits do not depend on which
      // part arrived last
      u32x4_t o[16];
      float2 ml1;
      load_part(u.first_slot + (u.slot == u.first_slot ? 1 : 0), o, ml1);
      const float M = fmaxf(m, ml1.x);
      const float Mu = M == -INFINITY ? 0.0f : M;
      const float a0 = exp2f(m - Mu), a1 = exp2f(ml1.x - Mu);
      add_part(o, a0, a1);
      {
#pragma clang fp contract(off)
        l = l * a0 + ml1.y * a1;
      }
    } else {
      // more parts: from zero, in part order (own partial re-read), a fixed
      // order whoever arrives last.  The common max first, from (m, l) loads
      // eight parts at a time (a short batch repeats the last part).
      float M = -INFINITY;
      for (int q0 = 0; q0 < np; q0 += 8) {
        float2 mb[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) mb[i] = load_ml(u.first_slot + min(q0 + i, np - 1));
#pragma unroll
        for (int i = 0; i < 8; ++i) M = fmaxf(M, mb[i].x);
      }
      const float Mu = M == -INFINITY ? 0.0f : M;
      l = 0.0f;
#pragma unroll
      for (int i = 0; i < 4; ++i) acc_o[i] = f32x16_t{};
      // then the parts in order, each part's loads in one batch
      for (int q = 0; q < np; ++q) {
        u32x4_t o[16];
        float2 mlq;
        load_part(u.first_slot + q, o, mlq);
        const float w = exp2f(mlq.x - Mu);
        add_part(o, 1.0f, w);
        l += mlq.y * w;
      }
    }
  }

  // ---- epilogue.  acc_o[dt] register r of lane (lq, g) holds O^T row
  // d = 32 dt + 8 (r/4) + 4 g + r%4, column = this lane's query.
  const float inv = l > 0.0f ? 1.0f / l : 0.0f;
  char* orow = p.o + ooff;
  if (p.dt_o == EA_BF16) {
    // Each wave stages its 32 rows in its own LDS region (the chunk
    // buffers are free after the walk's last barrier) and writes them as
    // 16-byte pieces of contiguous rows: the tile's rows are contiguous in
    // the O block, so every store instruction writes whole lines.
    constexpr int kPitch = 128 * 2 + 16;  // bytes per staged row
    char* stage = reinterpret_cast<char*>(sKV) + wq * 32 * kPitch;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int d = 32 * dt + 8 * rr + 4 * g;
        uint2 w;
        w.x = pack_bf16x2(acc_o[dt][4 * rr] * inv, acc_o[dt][4 * rr + 1] * inv);
        w.y = pack_bf16x2(acc_o[dt][4 * rr + 2] * inv, acc_o[dt][4 * rr + 3] * inv);
        *reinterpret_cast<uint2*>(stage + lq * kPitch + d * 2) = w;
      }
    const int64_t row0 = u.q0 + wq * 32;  // first row of this wave inside the block
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int c = k * 64 + lane, r = c >> 4, c16 = c & 15;
      const uint4 v = *reinterpret_cast<const uint4*>(stage + r * kPitch + c16 * 16);
      *reinterpret_cast<uint4*>(orow + ((row0 + r) * D + c16 * 8) * 2) = v;
    }
    return;
  }
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int d = 32 * dt + 8 * rr + 4 * g;
      const int64_t idx = (int64_t)row * D + d;
      const float o0 = acc_o[dt][4 * rr] * inv, o1 = acc_o[dt][4 * rr + 1] * inv;
      const float o2 = acc_o[dt][4 * rr + 2] * inv, o3 = acc_o[dt][4 * rr + 3] * inv;
      *reinterpret_cast<float4*>(orow + idx * 4) = make_float4(o0, o1, o2, o3);
    }
}

// Plan time: per unit, the Q and O blocks of its group and the K/V blocks of
// its run of tuples (one lane per tuple), from the GPU-built tuple table.
__global__ __launch_bounds__(64) void attn_prep_kernel(const AttnArgs p) {
  const AttnUnit u = p.units[blockIdx.x];
  const int32_t gb = p.goff[u.group], ge = p.goff[u.group + 1];
  const int n = ge - gb;
  const int tb = gb + (int)(((int64_t)u.part * n) / u.n_parts);
  const int te = gb + (int)(((int64_t)(u.part + 1) * n) / u.n_parts);
  AttnUnitMeta& um = p.meta[blockIdx.x];
  const int lane = threadIdx.x;
  if (lane == 0) {
    // every tuple of the group carries the same output and Q blocks
    const DevBlk& qb = p.blk_q[p.tuples[(int64_t)gb * 4 + 1]];
    um.qoff = qb.off;
    um.ooff = p.blk_o[p.tuples[(int64_t)gb * 4 + 0]].off;
    um.q_lo = qb.lo[p.q_dim];
    const int nt = min(te - tb, kAttnMaxUnitTuples);
    um.nt = nt;
    if (te - tb > kAttnMaxUnitTuples) *p.overflow = 1;  // the host refuses the plan
    // the walk's chunks: every kAttnChunkKeys keys of the unit's blocks, in
    // tuple order, up to the first chunk past the tile's last query (later
    // ones are masked for every row under the causal predicate)
    const int qpos_tile_min = qb.lo[p.q_dim] + u.q0, qpos_tile_max = qpos_tile_min + kAttnTileRows - 1;
    int nc = 0, n_plain = 0;
    bool plain = true;  // every chunk so far lies wholly before the tile's first query
    for (int t = 0; t < nt; ++t) {
      const DevBlk& kb = p.blk_k[p.tuples[(int64_t)(tb + t) * 4 + 2]];
      const int klo = kb.lo[p.k_dim], kext = kb.ext[p.k_dim];
      for (int c0 = 0; c0 < kext && !(p.causal && klo + c0 > qpos_tile_max); c0 += kAttnChunkKeys) {
        ++nc;
        plain = plain && !(p.causal && klo + c0 + kAttnChunkKeys - 1 > qpos_tile_min);
        n_plain += plain;
      }
    }
    um.nc = nc;
    um.n_plain = n_plain;
  }
  for (int t = lane; t < te - tb && t < kAttnMaxUnitTuples; t += 64) {
    const int32_t* tp = p.tuples + (int64_t)(tb + t) * 4;
    const DevBlk& kb = p.blk_k[tp[2]];
    AttnKv kv;
    kv.koff = kb.off;
    kv.voff = p.blk_v[tp[3]].off;
    kv.klo = kb.lo[p.k_dim];
    kv.kext = kb.ext[p.k_dim];
    um.kv[t] = kv;
  }
}

}  // namespace

hipError_t launch_attention_prep(const AttnArgs& a, hipStream_t s) {
  if (a.n_units == 0) return hipSuccess;
  hipLaunchKernelGGL(attn_prep_kernel, dim3((uint32_t)a.n_units), dim3(64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.n_units == 0) return hipSuccess;
  hipLaunchKernelGGL(attn_kernel, dim3((uint32_t)a.n_units), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace ea
