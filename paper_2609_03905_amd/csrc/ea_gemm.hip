// ea_gemm.hip -- block-GEMM join-agg on the CDNA4 matrix cores.
//
// Section 3.2, Example "Matrix multiply, decomposed": the per-tuple concrete
// operator is a block matrix product and the aggregation is +.  A workgroup
// owns a 256-row tile of one output block (one output key) and runs the
// K-loop over a run of that key's tuples, so the SUM of the partial products
// happens in the MFMA accumulators.  When an output key's tuples are split
// over several workgroups (to fill the 256 CUs), each writes its partial sum
// to the plan's scratch and the last one to arrive adds the partials in a
// fixed order (deterministic) and stores; otherwise the store is direct.  The
// recompose step is the store into the output block.
//
// Inputs bf16 or f16, fp32 accumulation (v_mfma_f32_32x32x16_{bf16,f16}).
// 512 threads = 8 waves in a 2 (rows) x 4 (columns) grid, two waves per SIMD
// so that one wave's LDS reads overlap the other's MFMAs.  Tile 256 x 256
// (each wave 128 x 64: 4 x 2 MFMA tiles, 128 accumulators), or 256 x 128
// (each wave 128 x 32), which a plan takes when 256-wide tiles would leave
// CUs idle or need split sums; for SwiGLU 256 x 128 with two right operands
// (each wave 128 x 32 per operand).
//
// Two K pipelines share the tile layout and the epilogue:
//   * gemm_dl_kernel (every contracted block extent a multiple of 32): operands
//     go straight from global memory into LDS (global_load_lds_dwordx4), four
//     stages of 32-deep K steps in flight, XOR-swizzled LDS chunks, [k][n]
//     right operands read with transposing LDS reads (description below);
//   * gemm_kernel (any 8-aligned extents): register-staged loads two K steps
//     ahead, K step 64, LDS double-buffered with padded rows; a right operand
//     stored [k][n] is transposed in registers before the LDS write.
//
// Epilogue: the tile is staged through LDS so that stores (and the residual
// loads) are 16-byte row chunks; the residual is added in fp32 before the one
// rounding to the output dtype; SwiGLU stores silu(g) * u of its two
// accumulators.
#include "ea_device.h"

namespace ea {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int TM = kGemmTM;  // 256
constexpr int TK = 64;
constexpr int PITCH = TK + 8;  // LDS row pitch in elements (144 bytes)

template <bool BF16>
__device__ __forceinline__ f32x16_t mfma(const uint4& a, const uint4& b, const f32x16_t& c) {
  if constexpr (BF16)
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                    __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, a),
                                                   __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
}

// 16-byte load that yields zeros when !ok.  The load always happens at an
// in-bounds address (the block base when masked; every block row on this
// path holds at least 16 bytes), so there is no branch and no pointer select.
__device__ __forceinline__ uint4 masked_load(const char* base, int64_t off, bool ok) {
  const uint4 v = *reinterpret_cast<const uint4*>(base + off);
  return ok ? v : make_uint4(0, 0, 0, 0);
}

__device__ __forceinline__ uint32_t word(const uint4& v, int w) {
  return w == 0 ? v.x : w == 1 ? v.y : w == 2 ? v.z : v.w;
}

// Uniform copy of a block's byte offset and 2-d extents (scalar loads).
struct BlkInfo {
  int64_t off;
  int e0, e1;
};

__device__ __forceinline__ BlkInfo blk_info(const DevBlk* tab, int32_t idx) {
  const DevBlk* b = tab + idx;
  return BlkInfo{ld_uniform(&b->off), ld_uniform(&b->ext[0]), ld_uniform(&b->ext[1])};
}

// ---- A tile: 256 rows x 64 k, k contiguous; 2048 16-byte pieces, NPA per thread
template <int T>
struct ATile {
  static constexpr int NPA = TM * TK / 8 / T;
  __device__ __forceinline__ static void load(uint4 (&r)[NPA], const char* base, const BlkInfo& ab, int m0, int k0,
                                              int tid) {
    const int mext = ab.e0, kext = ab.e1;
#pragma unroll
    for (int i = 0; i < NPA; ++i) {
      const int c = tid + T * i;
      const int gm = m0 + (c >> 3), gk = k0 + (c & 7) * 8;
      const bool ok = gm < mext && gk < kext;
      r[i] = masked_load(base, ok ? ((int64_t)gm * kext + gk) * 2 : 0, ok);
    }
  }
  __device__ __forceinline__ static void store(const uint4 (&r)[NPA], uint16_t* s, int tid) {
#pragma unroll
    for (int i = 0; i < NPA; ++i) {
      const int c = tid + T * i;
      *reinterpret_cast<uint4*>(s + (c >> 3) * PITCH + (c & 7) * 8) = r[i];
    }
  }
};

// ---- B tile: BN columns x 64 k, stored in LDS as [n][k].  [n][k] storage:
// NP = BN*64/8/T 16-byte pieces per thread.  [k][n] storage: blocks of
// 4 k x 8 n (block q: kg = q % 16, nc = q / 16), BN*64/32/T blocks per
// thread, rounded up (threads past the last block take none).
template <bool KMAJOR, int BN, int kThreads>
struct BTile {
  static constexpr int NBLK = BN * TK / 32;  // 4x8 blocks of the tile
  static constexpr int NP = KMAJOR ? BN * TK / 8 / kThreads : 4 * ((NBLK + kThreads - 1) / kThreads);
  __device__ __forceinline__ static void load(uint4 (&r)[NP], const char* base, const BlkInfo& bb, int n0, int k0,
                                              int tid) {
    if constexpr (!KMAJOR) {
      const int kext = bb.e0, next = bb.e1;
#pragma unroll
      for (int b = 0; b < NP / 4; ++b) {
        const int q = tid + kThreads * b;
        const int kg = q & 15, nc = q >> 4;
        const int gn = n0 + nc * 8;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int gk = k0 + kg * 4 + i;
          const bool ok = q < NBLK && gk < kext && gn < next;
          r[4 * b + i] = masked_load(base, ok ? ((int64_t)gk * next + gn) * 2 : 0, ok);
        }
      }
    } else {
      const int next = bb.e0, kext = bb.e1;
#pragma unroll
      for (int i = 0; i < NP; ++i) {
        const int c = tid + kThreads * i;
        const int gn = n0 + (c >> 3), gk = k0 + (c & 7) * 8;
        const bool ok = gn < next && gk < kext;
        r[i] = masked_load(base, ok ? ((int64_t)gn * kext + gk) * 2 : 0, ok);
      }
    }
  }
  __device__ __forceinline__ static void store(const uint4 (&r)[NP], uint16_t* s, int tid) {
    if constexpr (!KMAJOR) {
#pragma unroll
      for (int b = 0; b < NP / 4; ++b) {
        const int q = tid + kThreads * b;
        if (NBLK % kThreads != 0 && q >= NBLK) break;
        const int kg = q & 15, nc = q >> 4;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int w = j >> 1;
          const uint32_t x0 = word(r[4 * b], w), x1 = word(r[4 * b + 1], w);
          const uint32_t x2 = word(r[4 * b + 2], w), x3 = word(r[4 * b + 3], w);
          uint2 v;
          if ((j & 1) == 0) {
            v.x = (x0 & 0xffffu) | (x1 << 16);
            v.y = (x2 & 0xffffu) | (x3 << 16);
          } else {
            v.x = (x0 >> 16) | (x1 & 0xffff0000u);
            v.y = (x2 >> 16) | (x3 & 0xffff0000u);
          }
          *reinterpret_cast<uint2*>(s + (nc * 8 + j) * PITCH + kg * 4) = v;
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < NP; ++i) {
        const int c = tid + kThreads * i;
        *reinterpret_cast<uint4*>(s + (c >> 3) * PITCH + (c & 7) * 8) = r[i];
      }
    }
  }
};

struct EpiArgs {
  char* c;          // output block base
  const char* res;  // residual block base (same layout and dtype) or null
  int mext, next;   // output block extents
  int m0, n0;       // tile origin inside the block
};

// Epilogue through LDS.  Accumulator r of MFMA tile (i, j) in lane l holds
// row 8*(r/4) + 4*(l/32) + r%4 and column l%32 of that 32x32 tile, so a lane
// owns scattered 2-byte outputs.  The tile's values (SwiGLU: silu(g) * u) are
// therefore staged in LDS, in four passes of 64 rows (MFMA row-tile i of every
// wave), fp32 with a row pitch of kEpiPitch floats; then each thread takes 8
// consecutive columns of one row and stores them with one 16-byte access (two
// for fp32), reading the residual the same way.  Block rows are multiples of
// 8 elements on this path (host guarantee), so a chunk never straddles a row.
constexpr int kEpiPitch = 264;  // 256 + 8: rows 4 apart land on opposite halves of the 64 banks

template <bool SWIGLU, int NB, int WN, int W, int DT, bool RES>
__device__ __forceinline__ void epilogue(const f32x16_t (&acc)[NB][4][WN], const EpiArgs& e, float* stage,
                                         int wid, int lane) {
  constexpr int WGN = W / 2;            // waves along n (2 along m)
  constexpr int WCOLS = WN * 32;        // columns per wave
  constexpr int CPR = WGN * WCOLS / 8;  // 8-column chunks per tile row
  constexpr int CHUNKS = CPR / W;       // chunks per thread per pass (64 rows)
  static_assert(CPR % W == 0, "epilogue chunking");
  const int wm = wid / WGN, wn = wid % WGN, g = lane >> 5, lq = lane & 31;
  const int tid = wid * 64 + lane;
  // chunk k of pass i: tile row and 8-column group, global position
  auto chunk_pos = [&](int i, int k, int& row, int& c8, int& gm, int& gn) {
    const int c = tid + 64 * W * k;
    row = c / CPR;
    c8 = c % CPR;
    gm = e.m0 + (row >> 5) * 128 + 32 * i + (row & 31);
    gn = e.n0 + 8 * c8;
  };
  // A 16-bit residual is loaded for all four passes before the first one
  // (64 registers), so that one memory latency covers the whole epilogue
  // instead of one per pass; an fp32 residual is loaded pass by pass.
  constexpr bool RES16 = RES && DT != EA_F32;
  uint4 rres[RES16 ? 4 : 1][RES16 ? CHUNKS : 1];
  if constexpr (RES16) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int k = 0; k < CHUNKS; ++k) {
        int row, c8, gm, gn;
        chunk_pos(i, k, row, c8, gm, gn);
        rres[i][k] = gm < e.mext && gn < e.next
                         ? *reinterpret_cast<const uint4*>(e.res + ((int64_t)gm * e.next + gn) * 2)
                         : make_uint4(0, 0, 0, 0);
      }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    __syncthreads();  // the stage area is free (K loop or previous pass done)
#pragma unroll
    for (int j = 0; j < WN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float v = acc[0][i][j][r];
        // silu(g) * u: the reciprocal (about 1 ulp) in place of a correctly
        // rounded division, far below the output's bf16 rounding
        if constexpr (SWIGLU) v = v * __builtin_amdgcn_rcpf(1.0f + __expf(-v)) * acc[NB - 1][i][j][r];
        const int row = wm * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
        stage[row * kEpiPitch + wn * WCOLS + 32 * j + lq] = v;
      }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < CHUNKS; ++k) {
      int row, c8, gm, gn;
      chunk_pos(i, k, row, c8, gm, gn);
      if (gm < e.mext && gn < e.next) {
        const float4 lo = *reinterpret_cast<const float4*>(stage + row * kEpiPitch + 8 * c8);
        const float4 hi = *reinterpret_cast<const float4*>(stage + row * kEpiPitch + 8 * c8 + 4);
        float o[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        const int64_t idx = (int64_t)gm * e.next + gn;
        if constexpr (DT == EA_F32) {
          if constexpr (RES) {
            const float4 r0 = *reinterpret_cast<const float4*>(e.res + idx * 4);
            const float4 r1 = *reinterpret_cast<const float4*>(e.res + idx * 4 + 16);
            o[0] += r0.x; o[1] += r0.y; o[2] += r0.z; o[3] += r0.w;
            o[4] += r1.x; o[5] += r1.y; o[6] += r1.z; o[7] += r1.w;
          }
          *reinterpret_cast<float4*>(e.c + idx * 4) = make_float4(o[0], o[1], o[2], o[3]);
          *reinterpret_cast<float4*>(e.c + idx * 4 + 16) = make_float4(o[4], o[5], o[6], o[7]);
        } else {
          if constexpr (RES) {
            const uint4 rv = rres[i][k];
            const uint32_t w[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const uint16_t h0 = (uint16_t)(w[q] & 0xffffu), h1 = (uint16_t)(w[q] >> 16);
              o[2 * q] += DT == EA_BF16 ? bf16_to_f32(h0) : f16_to_f32(h0);
              o[2 * q + 1] += DT == EA_BF16 ? bf16_to_f32(h1) : f16_to_f32(h1);
            }
          }
          uint32_t w[4];
#pragma unroll
          for (int q = 0; q < 4; ++q)
            w[q] = DT == EA_BF16 ? pack_bf16x2(o[2 * q], o[2 * q + 1])
                                 : (uint32_t)f32_to_f16(o[2 * q]) | ((uint32_t)f32_to_f16(o[2 * q + 1]) << 16);
          *reinterpret_cast<uint4*>(e.c + idx * 2) = make_uint4(w[0], w[1], w[2], w[3]);
        }
      }
    }
  }
}

// Position of a K step: tuple index and offset inside its contracted block.
struct KStep {
  int t, k0;
};

// Split output keys of three or more parts: every unit writes its partial
// sums, and the last unit of the key to arrive (device-scope arrival counter)
// adds the partials in part order from zero and stores.
// Two parts: the first to arrive writes its partial and marks it written;
// the second keeps its own in registers, waits for that mark and merges, so
// one partial per tile is written instead of two.  The second arriver waits
// only for a workgroup that has already arrived, i.e. is running and only
// storing, so the wait ends within that store's time (a few us); the 100 ms
// guard could only be reached by a writer descheduled for that long.  Its
// sum, own + other, equals other + own exactly, so the result does not depend
// on which part arrived first.
// Partials are laid out in accumulator order (lane-contiguous float4s).
// Then the epilogue, with dtype and residual decided outside its unrolled loops.
constexpr int32_t kWritten = 1 << 16;         // added by the first of two parts once its partial is stored
constexpr uint64_t kWrittenWaitTicks = 10000000;  // guard on the second's wait: 100 ms of the 100 MHz clock
template <bool SWIGLU, int NB, int WN, int W>
__device__ __forceinline__ void finish_tile(f32x16_t (&acc)[NB][4][WN], const GemmArgs& p, const GemmTile& tile,
                                            int wid, int lane, float* stage) {
  __shared__ int s_last;
  const int tid = wid * 64 + lane;
  if (tile.n_parts > 1) {
    // Partial sums go through the plan's scratch as lane-contiguous 16-byte
    // pieces (every store instruction writes whole 128-byte lines) with the
    // sc1 cache policy, which keeps them coherent between the XCDs' L2s; the
    // reader's loads carry it too.  Every lane holds PER_WAVE floats.
    constexpr int PER_WAVE = NB * 4 * WN * 16;
    constexpr int WAVE_BYTES = PER_WAVE * 64 * 4;
    constexpr int kCoherent = 16;  // sc1
    auto slot_rsrc = [&](int slot) {
      return __builtin_amdgcn_make_buffer_rsrc(p.partials + (int64_t)slot * W * PER_WAVE * 64, 0, 0x7fffffff,
                                               0x00020000);
    };
    auto piece = [&](int o, int i, int j, int r4) {  // byte offset of a lane's piece in its wave's area
      const int q = ((o * 4 + i) * WN + j) * 4 + r4;
      return (uint32_t)(wid * WAVE_BYTES + (q * 64 + lane) * 16);
    };
    int32_t* const counter = p.counters + tile.counter;
    // two parts: arrivals in the low bits; the second sees 1, or
    // 1 + kWritten when the first has already stored its partial
    const bool two_parts = tile.n_parts == 2;
    bool write = true;
    if (two_parts) {
      if (tid == 0) s_last = (arrive_agent(counter) & (kWritten - 1)) == 1;
      __syncthreads();
      write = !s_last;
    }
    if (write) {
      const auto rs = slot_rsrc(tile.slot);
#pragma unroll
      for (int o = 0; o < NB; ++o)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < WN; ++j)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
              const f32x16_t& c = acc[o][i][j];
              const u32x4_t v = {__float_as_uint(c[4 * r4]), __float_as_uint(c[4 * r4 + 1]),
                                 __float_as_uint(c[4 * r4 + 2]), __float_as_uint(c[4 * r4 + 3])};
              __builtin_amdgcn_raw_buffer_store_b128(v, rs, piece(o, i, j, r4), 0, kCoherent);
            }
      drain_vmem();
    }
    __syncthreads();
    if (tid == 0) {
      if (!two_parts) {
        s_last = arrive_agent(counter) == tile.n_parts - 1;
      } else if (write) {
        __hip_atomic_fetch_add(counter, kWritten, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      } else {  // the first arriver is storing: wait for its mark
        const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
        while (__hip_atomic_load(counter, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < kWritten &&
               __builtin_amdgcn_s_memrealtime() - t0 < kWrittenWaitTicks)
          __builtin_amdgcn_s_sleep(2);
      }
    }
    __syncthreads();
    if (!s_last) return;
    // add one slot's partials: 16 loads in flight per batch (latency hidden,
    // 64 registers), then their adds
    auto add_slot = [&](int slot) {
      const auto rs = slot_rsrc(slot);
      constexpr int NQ = PER_WAVE / 4, BATCH = 16;
      static_assert(NQ % BATCH == 0, "batches of pieces");
#pragma unroll
      for (int q0 = 0; q0 < NQ; q0 += BATCH) {
        u32x4_t v[BATCH];
#pragma unroll
        for (int t = 0; t < BATCH; ++t) {
          const int q = q0 + t;
          v[t] = __builtin_amdgcn_raw_buffer_load_b128(rs, piece(q / (16 * WN), (q / (4 * WN)) % 4, (q / 4) % WN, q % 4),
                                                       0, kCoherent);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int t = 0; t < BATCH; ++t) {
          const int q = q0 + t;
          f32x16_t& c = acc[q / (16 * WN)][(q / (4 * WN)) % 4][(q / 4) % WN];
          const int r4 = q % 4;
          c[4 * r4] += __uint_as_float(v[t].x);
          c[4 * r4 + 1] += __uint_as_float(v[t].y);
          c[4 * r4 + 2] += __uint_as_float(v[t].z);
          c[4 * r4 + 3] += __uint_as_float(v[t].w);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    // Two parts: own + other, and a + b == b + a exactly, so the result does
    // not depend on which part arrived last and our own partial is not
    // reloaded.  More parts: the sum in part order from zero, a fixed order
    // whoever arrives last.
    const bool two = tile.n_parts == 2;
    const int other = tile.first_slot + (tile.slot == tile.first_slot ? 1 : 0);
    if (!two) {
#pragma unroll
      for (int o = 0; o < NB; ++o)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < WN; ++j) acc[o][i][j] = f32x16_t{};
    }
    const int n_add = two ? 1 : tile.n_parts;
    for (int k = 0; k < n_add; ++k) add_slot(two ? other : tile.first_slot + k);
    if (tid == 0) reset_agent(counter);  // ready for the next call (stream-ordered)
  }
  const DevBlk& cb = p.blk_c[tile.block];
  const EpiArgs e{p.c + cb.off, p.res ? p.res + cb.off : nullptr, cb.ext[0], cb.ext[1], tile.m0, tile.n0};
  if (!e.res && p.dt_out == EA_BF16) epilogue<SWIGLU, NB, WN, W, EA_BF16, false>(acc, e, stage, wid, lane);
  else if (!e.res && p.dt_out == EA_F32) epilogue<SWIGLU, NB, WN, W, EA_F32, false>(acc, e, stage, wid, lane);
  else if (p.dt_out == EA_BF16) epilogue<SWIGLU, NB, WN, W, EA_BF16, true>(acc, e, stage, wid, lane);
  else if (p.dt_out == EA_F32) epilogue<SWIGLU, NB, WN, W, EA_F32, true>(acc, e, stage, wid, lane);
  else if (!e.res) epilogue<SWIGLU, NB, WN, W, EA_F16, false>(acc, e, stage, wid, lane);
  else epilogue<SWIGLU, NB, WN, W, EA_F16, true>(acc, e, stage, wid, lane);
}

template <bool BF16, bool KMAJOR, bool SWIGLU, int W>
__global__ __launch_bounds__(W * 64, 1) void gemm_kernel(const GemmArgs p) {
  constexpr int kThreads = W * 64;
  constexpr int NB = SWIGLU ? 2 : 1;      // right operands
  constexpr int BN = SWIGLU ? 128 : 256;  // columns per right operand
  constexpr int WGN = W / 2;              // waves along n (2 along m)
  constexpr int WCOLS = BN / WGN;         // columns per wave, per operand
  constexpr int WN = WCOLS / 32;          // MFMA tiles per wave along n, per operand
  using BT = BTile<KMAJOR, BN, kThreads>;
  using AT = ATile<kThreads>;
  constexpr int NPA = AT::NPA;
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][TM * PITCH];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][NB * BN * PITCH];

  // kernel arguments into registers (no address of the argument block is taken)
  const int32_t* __restrict__ tuples = p.tuples;
  const DevBlk* __restrict__ blk_a = p.blk_a;
  const DevBlk* __restrict__ blk_b = p.blk_b;
  const DevBlk* __restrict__ blk_b2 = p.blk_b2;
  const char* __restrict__ pa = p.a;
  const char* __restrict__ pb = p.b;
  const char* __restrict__ pb2 = p.b2;
  const int ts = p.tuple_stride;

  const GemmTile tile = ld_uniform(p.tiles + blockIdx.x);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid / WGN, wn = wid % WGN;
  const int g = lane >> 5, lq = lane & 31;
  const int32_t gb = ld_uniform(p.goff + tile.block), ge = ld_uniform(p.goff + tile.block + 1);
  const int n_t = ge - gb;
  const int t_begin = gb + (int)(((int64_t)tile.part * n_t) / tile.n_parts);
  const int t_end = gb + (int)(((int64_t)(tile.part + 1) * n_t) / tile.n_parts);

  f32x16_t acc[NB][4][WN];
#pragma unroll
  for (int o = 0; o < NB; ++o)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < WN; ++j) acc[o][i][j] = f32x16_t{};

  auto advance = [&](KStep st) -> KStep {
    st.k0 += TK;
    if (st.k0 >= ld_uniform(&blk_a[ld_uniform(tuples + (int64_t)st.t * ts + 1)].ext[1])) {
      st.t += 1;
      st.k0 = 0;
    }
    return st;
  };
  // two register stages of prefetched operands
  uint4 ra[2][NPA], rb[2][NB][BT::NP];
  auto load_step = [&](int set, KStep st) {
    const int32_t* tp = tuples + (int64_t)st.t * ts;
    const BlkInfo ab = blk_info(blk_a, ld_uniform(tp + 1));
    AT::load(ra[set], pa + ab.off, ab, tile.m0, st.k0, tid);
    const BlkInfo bb = blk_info(blk_b, ld_uniform(tp + 2));
    BT::load(rb[set][0], pb + bb.off, bb, tile.n0, st.k0, tid);
    if constexpr (SWIGLU) {
      const BlkInfo bb2 = blk_info(blk_b2, ld_uniform(tp + 3));
      BT::load(rb[set][NB - 1], pb2 + bb2.off, bb2, tile.n0, st.k0, tid);
    }
  };
  auto store_step = [&](int set, int buf) {
    AT::store(ra[set], sA[buf], tid);
#pragma unroll
    for (int o = 0; o < NB; ++o) BT::store(rb[set][o], sB[buf] + o * BN * PITCH, tid);
  };
  auto compute = [&](int buf) {
    const uint16_t* a_s = sA[buf] + (wm * 128 + lq) * PITCH + 8 * g;
    const uint16_t* b_s = sB[buf] + (wn * WCOLS + lq) * PITCH + 8 * g;
#pragma unroll
    for (int s = 0; s < TK / 16; ++s) {
      uint4 af[4], bf[NB][WN];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const uint4*>(a_s + i * 32 * PITCH + s * 16);
#pragma unroll
      for (int o = 0; o < NB; ++o)
#pragma unroll
        for (int j = 0; j < WN; ++j)
          bf[o][j] = *reinterpret_cast<const uint4*>(b_s + (o * BN + j * 32) * PITCH + s * 16);
#pragma unroll
      for (int o = 0; o < NB; ++o)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < WN; ++j) acc[o][i][j] = mfma<BF16>(af[i], bf[o][j], acc[o][i][j]);
    }
  };

  // Pipeline: step s is computed from LDS buffer s%2; its operands were
  // stored there at the end of step s-1 from register set s%2, which was
  // loaded during step s-2.
  KStep cur{t_begin, 0};
  if (cur.t < t_end) {
    load_step(0, cur);
    KStep nx = advance(cur);
    if (nx.t < t_end) load_step(1, nx);
    store_step(0, 0);
  }
  __syncthreads();
  // unrolled by two so that register sets are indexed statically
  while (cur.t < t_end) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (cur.t >= t_end) break;
      const KStep n1 = advance(cur);
      const KStep n2 = n1.t < t_end ? advance(n1) : n1;
      if (n2.t < t_end) load_step(h, n2);      // two steps ahead, into the set just consumed
      compute(h);
      if (n1.t < t_end) store_step(h ^ 1, h ^ 1);
      __syncthreads();
      cur = n1;
    }
  }

  static_assert(sizeof(sA) >= 64 * kEpiPitch * sizeof(float), "epilogue stage");
  finish_tile<SWIGLU, NB, WN, W>(acc, p, tile, wid, lane, reinterpret_cast<float*>(&sA[0][0]));
}

// ===========================================================================
// Direct-to-LDS pipeline (fast path): operands go from global memory straight
// into LDS (global_load_lds, 16 bytes per lane, lane-linear placement), with
// no staging registers and no LDS write instructions.  Four stages of 32-deep
// K steps (4 x 32 KiB) keep three steps of loads in flight while one is
// computed.  LDS layouts, 16-byte chunks XOR-swizzled so that the fragment
// reads are free of bank conflicts.  The LDS has 64 four-byte banks; a
// ds_read_b128 is served 16 lanes per cycle, and the 16 lanes of one cycle are
// four lane quads (4 consecutive lanes) of one half-wave with the same parity
// of lane bits 2..4 (lanes 0-3, 12-15, 20-23, 24-27 together, and so on;
// measured with the LDS bank-conflict counter), so those 16 lanes must read
// 16 distinct 16-byte positions modulo 256 bytes:
//   A, and B stored [n][k]: row r (64 bytes = 4 chunks), logical chunk c at
//     physical chunk c ^ swz_row(r);
//   B stored [k][n]: row k (BN*2 bytes), logical chunk c at physical chunk
//     c ^ swz_k(k); the MFMA operand (8 consecutive k of one column) is
//     read with two ds_read_b64_tr_b16: in each 16-lane group, lane 4k'+r
//     reads 4 columns N0+4r.. of row K0+k', and lane i receives rows K0..K0+3
//     of column N0+i.
// Rows or columns past a block's edge load from the block base instead (their
// products land only in accumulator rows/columns that are never stored); the
// K extent of every contracted block must be a multiple of 32.
// ===========================================================================
constexpr int DK = 32;  // K per stage
constexpr int NSTAGE = 4;

typedef short s16x4 __attribute__((ext_vector_type(4)));

// 64-byte rows: a fragment read gives lane l row l % 32 and one logical
// chunk for the half-wave.  The four lanes of a quad take the four row
// positions mod 256 bytes; the four quads of one read cycle differ in row
// bits 2..3 (their quad indices, 0 3 5 6 or 1 2 4 7, are distinct mod 4), so
// XOR-ing those bits into the chunk gives each quad its own chunk column.
__device__ __forceinline__ int swz_row(int r) { return (r >> 2) & 3; }
// [k][n] rows (a multiple of 256 bytes): the 4 k rows of one transposed read
// take disjoint chunk sets, for each half of the 32 lanes and for all 32.
__device__ __forceinline__ int swz_k(int k) { return (2 * (k & 3)) ^ (8 * (k & 1)); }

// One direct global->LDS load: each lane fetches 16 bytes at base + voff and
// the wave's 64 pieces land contiguously at LDS byte address lds_addr
// (lane-linear).  The base is wave-uniform (scalar registers) and the lane
// offset 32-bit: the load path takes this form at a markedly higher rate
// than 64-bit per-lane addresses.  Issued through inline asm so that the
// compiler does not track the LDS write: the kernel orders it explicitly
// (vmcnt wait for the stage, then a barrier), and the compiler's own
// in-order vmcnt waits stay correct (later loads only make them more
// conservative).
__device__ __forceinline__ void dl_load16(const char* base, uint32_t voff, uint32_t lds_addr) {
  const uint32_t lds = __builtin_amdgcn_readfirstlane(lds_addr);  // wave-uniform
  // both halves of the base made uniform as unsigned 32-bit values (a signed
  // readfirstlane result would be sign-extended when widened)
  const uint64_t b = (uint64_t)(uintptr_t)base;
  const uint32_t b_lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b);
  const uint32_t b_hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
  const uint64_t sbase = (uint64_t)b_lo | ((uint64_t)b_hi << 32);
  // M0 is listed as clobbered; nothing else in these kernels reads M0 (no
  // LDS-parameter, message or relative-move instructions), so the warning
  // that clang gives for a reserved register is silenced here.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
#pragma clang diagnostic pop
}

__device__ __forceinline__ uint2 tr_read(const uint16_t* p) {
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)p);
  return __builtin_bit_cast(uint2, v);
}

// vmcnt waits (gfx9 encoding: vmcnt bits [3:0] and [15:14], expcnt [6:4] and
// lgkmcnt [11:8] left at their maxima)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// The group's per-tuple operand metadata (GemmTupleMeta, resolved at plan
// time) is staged in LDS before the pipeline starts, so that the K loop reads
// it (once per tuple) with LDS reads and never with vector-memory loads,
// which share a counter with the in-flight operand loads.

// Workgroup barrier for the direct-load pipeline.  __syncthreads() carries a
// workgroup-scope fence that waits for every outstanding LDS-DMA load, which
// would drain the prefetch; here the stage's own loads are already waited for
// (vmcnt), so only this wave's LDS reads must finish (lgkmcnt) before the
// barrier.  The scheduling barriers keep the compiler from moving any
// instruction (memory or MFMA) across it.
__device__ __forceinline__ void stage_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((15) | (3 << 14) | (7 << 4) | (0 << 8));  // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

template <bool BF16, bool KMAJOR, bool SWIGLU, bool NARROW, int W>
__global__ __launch_bounds__(64 * W, 1) void gemm_dl_kernel(const GemmArgs p) {
  constexpr int WGN = W / 2;                         // waves along n (2 along m)
  constexpr int NB = SWIGLU ? 2 : 1;                 // right operands
  constexpr int BN = SWIGLU || NARROW ? 128 : 256;  // columns per right operand
  constexpr int WCOLS = BN / WGN;              // columns per wave, per operand
  constexpr int WN = WCOLS / 32;               // MFMA tiles per wave along n, per operand
  constexpr int A_ELEMS = TM * DK;             // per stage
  constexpr int B_ELEMS = BN * DK;             // per stage and right operand
  constexpr int STAGE = A_ELEMS + NB * B_ELEMS;
  constexpr int LA = A_ELEMS * 2 / 1024 / W;   // direct loads per wave and stage: A
  constexpr int LBO = B_ELEMS * 2 / 1024 / W;  // ... and each right operand
  constexpr int LS = LA + NB * LBO;
  constexpr int ROWB = BN * 2;                 // bytes per k row of a [k][n] B stage
  constexpr int RPI = 1024 / ROWB;             // [k][n] rows per load instruction
  constexpr int CPR = ROWB / 16;               // 16-byte chunks per [k][n] row
  static_assert(LA >= 1 && LBO >= 1 && 4 * LS < 64, "stage shape");
  __shared__ __attribute__((aligned(1024))) uint16_t smem[NSTAGE * STAGE];
  __shared__ GemmTupleMeta s_meta[kGemmMaxTuples];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid / WGN, wn = wid % WGN;
  const int g = lane >> 5, lq = lane & 31;
  const GemmUnit* unit = p.units + blockIdx.x;
  // the unit's segments, each run by the same straight-line code (two calls
  // rather than a loop, which would keep more registers live and spill)
  auto run_segment = [&](const GemmSeg& seg) __attribute__((always_inline)) {
  GemmTile tile;
  tile.block = seg.block;
  tile.m0 = seg.m0;
  tile.n0 = seg.n0;
  tile.part = seg.part;
  tile.n_parts = seg.n_parts;
  tile.slot = seg.first_slot + seg.part;
  tile.first_slot = seg.first_slot;
  tile.counter = seg.counter;
  // the group's tuples [gb, gb + nt), nt <= kGemmMaxTuples (host guarantee),
  // resolved from the join at plan time: one load per tuple, no chain of
  // dependent table lookups at the start of the kernel
  const int gb = seg.gb, nt = seg.nt;
  for (int i = tid; i < nt; i += 64 * W) s_meta[i] = p.meta[gb + i];
  __syncthreads();

  f32x16_t acc[NB][4][WN];
#pragma unroll
  for (int o = 0; o < NB; ++o)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < WN; ++j) acc[o][i][j] = f32x16_t{};

  // the segment's K steps [s0, s1) of the walk over the group's tuples (every
  // contracted block extent is a multiple of DK), from the plan: the step
  // count (never past the group's last step), the tuple holding step s0 and
  // how many of its steps come before s0
  const int n_steps = seg.n_steps;
  int it_t = seg.t0, skip = seg.skip;

  // ---- direct-load walk over the unit's K steps.  Per tuple, each operand
  // block has a uniform base address and each lane a 32-bit byte offset per
  // load instruction (every operand block is smaller than 4 GiB, a host
  // guarantee); a K step advances the offsets by a uniform stride.  Rows (A,
  // [n][k] B) or columns ([k][n] B) past a block's edge read row 0 / column 0
  // of the block instead, which stays in bounds for every K step of the block.
  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint16_t*)smem;
  const char* a_base = p.a;
  const char* b_base[NB];
  uint32_t va[LA], vb[NB][LBO];
  uint32_t bstep[NB];
  int left = 0;
  auto set_tuple = [&](int t) {
    const GemmTupleMeta& m = s_meta[t];
    a_base = p.a + m.aoff;
#pragma unroll
    for (int q = 0; q < LA; ++q) {
      const int r = (wid * LA + q) * 16 + (lane >> 2);
      const int c = (lane & 3) ^ swz_row(r);
      const int gm = tile.m0 + r;
      va[q] = (uint32_t)(((gm < m.am ? (int64_t)gm * m.ak : 0) + 8 * c) * 2);
    }
#pragma unroll
    for (int o = 0; o < NB; ++o) {
      b_base[o] = o == 0 ? p.b + m.boff : p.b2 + m.b2off;
      const int e0 = o == 0 ? m.b0 : m.b20, e1 = o == 0 ? m.b1 : m.b21;
      if constexpr (KMAJOR) {  // [n][k]: like A, BN rows of DK k
#pragma unroll
        for (int q = 0; q < LBO; ++q) {
          const int r = (wid * LBO + q) * 16 + (lane >> 2);
          const int c = (lane & 3) ^ swz_row(r);
          const int gn = tile.n0 + r;
          vb[o][q] = (uint32_t)(((gn < e0 ? (int64_t)gn * e1 : 0) + 8 * c) * 2);
        }
        bstep[o] = DK * 2;
      } else {  // [k][n]: DK rows of BN columns
#pragma unroll
        for (int q = 0; q < LBO; ++q) {
          const int k = (wid * LBO + q) * RPI + lane / CPR;
          const int c = (lane % CPR) ^ swz_k(k);
          const int gn = tile.n0 + 8 * c;
          vb[o][q] = (uint32_t)(((int64_t)k * e1 + (gn < e1 ? gn : 0)) * 2);
        }
        bstep[o] = (uint32_t)(DK * e1 * 2);
      }
    }
    left = m.ak / DK;
  };
  auto seek = [&]() {  // first tuple at or after it_t with a K step
    while (it_t < nt && s_meta[it_t].ak < DK) ++it_t;
    if (it_t < nt) set_tuple(it_t);
  };
  // issue the loads of the next K step of the walk into stage u
  auto issue_next = [&](int u) {
    const uint32_t sbase = lds_base + (uint32_t)(u * STAGE * 2);
#pragma unroll
    for (int q = 0; q < LA; ++q) {
      dl_load16(a_base, va[q], sbase + (uint32_t)((wid * LA + q) * 1024));
      va[q] += DK * 2;
    }
#pragma unroll
    for (int o = 0; o < NB; ++o)
#pragma unroll
      for (int q = 0; q < LBO; ++q) {
        dl_load16(b_base[o], vb[o][q], sbase + (uint32_t)(A_ELEMS * 2 + o * B_ELEMS * 2 + (wid * LBO + q) * 1024));
        vb[o][q] += bstep[o];
      }
    if (--left == 0) {
      ++it_t;
      seek();
    }
  };

  // ---- MFMA operands of one 16-deep half of a stage
  struct Frag {
    uint4 a[4];
    uint4 b[NB][WN];
  };
  auto load_frag = [&](Frag& f, int u, int s) {
    const uint16_t* sa = smem + u * STAGE;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = wm * 128 + i * 32 + lq;
      const int c = (2 * s + g) ^ swz_row(r);
      f.a[i] = *reinterpret_cast<const uint4*>(sa + r * DK + 8 * c);
    }
#pragma unroll
    for (int o = 0; o < NB; ++o)
#pragma unroll
      for (int j = 0; j < WN; ++j) {
        const uint16_t* sbo = sa + A_ELEMS + o * B_ELEMS;
        if constexpr (KMAJOR) {
          const int r = wn * WCOLS + j * 32 + lq;
          const int c = (2 * s + g) ^ swz_row(r);
          f.b[o][j] = *reinterpret_cast<const uint4*>(sbo + r * DK + 8 * c);
        } else {
          const int gq = lane >> 4, li = lane & 15;
          const int n = wn * WCOLS + j * 32 + 16 * (gq & 1) + 4 * (li & 3);
          uint2 h2[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int k = 16 * s + 8 * (gq >> 1) + 4 * h + (li >> 2);
            const int c = (n >> 3) ^ swz_k(k);
            h2[h] = tr_read(sbo + k * BN + 8 * c + (n & 4));
          }
          f.b[o][j] = make_uint4(h2[0].x, h2[0].y, h2[1].x, h2[1].y);
        }
      }
  };
  auto mma = [&](const Frag& f) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int o = 0; o < NB; ++o)
#pragma unroll
        for (int j = 0; j < WN; ++j) acc[o][i][j] = mfma<BF16>(f.a[i], f.b[o][j], acc[o][i][j]);
  };

  // ---- ping-pong pipeline.  Waves 0-3 (rows 0-127 of the tile, one wave
  // per SIMD) and waves 4-7 (rows 128-255) alternate between a memory phase
  // and a compute phase, with a workgroup barrier between phases and waves
  // 4-7 one phase behind.  So on every SIMD one wave issues the 16 MFMAs of a
  // 32-deep step while the other reads its operands of the step from LDS and
  // issues its share of the direct loads D steps ahead: the matrix core is
  // never left waiting for two waves that load at the same time.
  //   memory phase of step k: issue step k+D into the stage of step k-1
  //     (every read of that stage finished before the previous barrier),
  //     read stage k into registers, wait for this wave's loads of step k+1
  //     (waves 4-7; waves 0-3 wait after their compute phase), barrier.
  //     The loads go first: they hold the wave on the load path's address
  //     rate, and the operand reads queued behind them still land before
  //     the barrier (measured: 2-4% faster than reads first; loads placed
  //     between the MFMAs stall the compute phase instead);
  //   compute phase of step k: 16 MFMAs, barrier.
  // A stage is read only after every wave has waited for its own loads of
  // it and then passed a barrier; a stage is refilled only after both
  // groups' reads of it completed (lgkmcnt 0) before a barrier.
  constexpr int D = NSTAGE - 1;
  static_assert(D == 3, "vmcnt waits below cover up to two later steps");
  const int grp = wid / WGN;
  auto wait_after = [&](int later) {  // this wave's loads of a step landed; `later` steps issued after it
    if (later >= 2) wait_vmcnt<2 * LS>();
    else if (later == 1) wait_vmcnt<LS>();
    else wait_vmcnt<0>();
  };
  seek();
  if (skip > 0 && it_t < nt) {  // start inside the tuple: advance past its first `skip` steps
#pragma unroll
    for (int q = 0; q < LA; ++q) va[q] += (uint32_t)(skip * DK * 2);
#pragma unroll
    for (int o = 0; o < NB; ++o)
#pragma unroll
      for (int q = 0; q < LBO; ++q) vb[o][q] += (uint32_t)skip * bstep[o];
    left -= skip;
  }
  const int n_pro = n_steps < D ? n_steps : D;
  for (int st = 0; st < n_pro; ++st) issue_next(st);
  if (n_steps > 0) {
    wait_after(n_pro - 1);
    stage_barrier();
    if (grp == 1) stage_barrier();  // waves 4-7 start one phase behind
    Frag f0, f1;
    for (int k = 0; k < n_steps; ++k) {
      const int u = k % NSTAGE;
      if (k + D < n_steps) issue_next((k + D) % NSTAGE);
      load_frag(f0, u, 0);
      load_frag(f1, u, 1);
      const int later = (k + D < n_steps ? k + D : n_steps - 1) - (k + 1);
      if (grp == 1 && k + 1 < n_steps) wait_after(later);
      stage_barrier();  // lgkmcnt(0): operands in registers, stage u read
      mma(f0);
      mma(f1);
      if (grp == 0 && k + 1 < n_steps) wait_after(later);
      stage_barrier();
    }
    if (grp == 0) stage_barrier();  // ... and waves 0-3 end one phase early
  }
  static_assert(sizeof(smem) >= 64 * kEpiPitch * sizeof(float), "epilogue stage");
  finish_tile<SWIGLU, NB, WN, W>(acc, p, tile, wid, lane, reinterpret_cast<float*>(smem));
  };
  run_segment(unit->seg[0]);
  if (unit->n_seg > 1) {
    drain_vmem();  // the first segment's epilogue is done with its stores and the LDS
    __syncthreads();
    run_segment(unit->seg[1]);
  }
}

template <bool BF16, bool KMAJOR, bool SWIGLU>
hipError_t launch3(const GemmArgs& a, hipStream_t s) {
  if (a.direct && !SWIGLU && a.tile_n == 128)
    hipLaunchKernelGGL((gemm_dl_kernel<BF16, KMAJOR, false, true, 8>), dim3((uint32_t)a.n_units), dim3(512), 0, s, a);
  else if (a.direct)
    hipLaunchKernelGGL((gemm_dl_kernel<BF16, KMAJOR, SWIGLU, false, 8>), dim3((uint32_t)a.n_units), dim3(512), 0, s,
                       a);
  else
    hipLaunchKernelGGL((gemm_kernel<BF16, KMAJOR, SWIGLU, 8>), dim3((uint32_t)a.n_tiles), dim3(512), 0, s, a);
  return hipGetLastError();
}

template <bool BF16, bool KMAJOR>
hipError_t launch2(const GemmArgs& a, hipStream_t s) {
  return a.swiglu ? launch3<BF16, KMAJOR, true>(a, s) : launch3<BF16, KMAJOR, false>(a, s);
}

template <bool BF16>
hipError_t launch1(const GemmArgs& a, hipStream_t s) {
  return a.b_kmajor ? launch2<BF16, true>(a, s) : launch2<BF16, false>(a, s);
}

// Plan time, after the join.  One thread per tuple of the join: its operand
// blocks' offsets and extents, in tuple-table order.
__global__ __launch_bounds__(256) void gemm_meta_kernel(const GemmArgs p, int64_t tuple_cap) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= tuple_cap || q >= *p.count) return;
  const int32_t* tp = p.tuples + q * p.tuple_stride;
  const DevBlk& ab = p.blk_a[tp[1]];
  const DevBlk& bb = p.blk_b[tp[2]];
  GemmTupleMeta m;
  m.aoff = ab.off;
  m.am = ab.ext[0];
  m.ak = ab.ext[1];
  m.boff = bb.off;
  m.b0 = bb.ext[0];
  m.b1 = bb.ext[1];
  if (p.swiglu) {
    const DevBlk& b2 = p.blk_b2[tp[3]];
    m.b2off = b2.off;
    m.b20 = b2.ext[0];
    m.b21 = b2.ext[1];
  } else {
    m.b2off = 0;
    m.b20 = m.b21 = 0;
  }
  m.pad[0] = m.pad[1] = m.pad[2] = m.pad[3] = 0;
  p.meta[q] = m;
}

// Plan time, after the join.  One thread per unit: each segment's group
// (first tuple, count) and where its K steps start in the group's walk.
__global__ __launch_bounds__(256) void gemm_seg_kernel(const GemmArgs p, GemmUnit* units) {
  const int u = blockIdx.x * 256 + threadIdx.x;
  if (u >= p.n_units) return;
  GemmUnit& un = units[u];
  for (int k = 0; k < un.n_seg && k < kGemmMaxSegs; ++k) {
    GemmSeg& sg = un.seg[k];
    const int32_t gb = p.goff[sg.block], nt = p.goff[sg.block + 1] - gb;
    auto steps = [&](int i) { return p.blk_a[p.tuples[(int64_t)(gb + i) * p.tuple_stride + 1]].ext[1] / DK; };
    int group_steps = 0;
    for (int i = 0; i < nt; ++i) group_steps += steps(i);
    int t = 0, skip = sg.s0;
    while (t < nt && skip >= steps(t)) {
      skip -= steps(t);
      ++t;
    }
    sg.gb = gb;
    sg.nt = nt;
    sg.t0 = t;
    sg.skip = skip;
    sg.n_steps = max(0, min(sg.s1, group_steps) - sg.s0);  // never past the group's last step
  }
}

}  // namespace

hipError_t launch_gemm_prep(const GemmArgs& a, GemmUnit* units, int64_t tuple_cap, hipStream_t s) {
  if (tuple_cap > 0)
    hipLaunchKernelGGL(gemm_meta_kernel, dim3((uint32_t)((tuple_cap + 255) / 256)), dim3(256), 0, s, a, tuple_cap);
  if (a.n_units > 0)
    hipLaunchKernelGGL(gemm_seg_kernel, dim3((uint32_t)((a.n_units + 255) / 256)), dim3(256), 0, s, a, units);
  return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs& a, hipStream_t s) {
  if ((a.direct ? a.n_units : a.n_tiles) == 0) return hipSuccess;
  return a.dt_in == EA_BF16 ? launch1<true>(a, s) : launch1<false>(a, s);
}

}  // namespace ea
