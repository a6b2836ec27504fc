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
// 256 threads = 4 waves in a 2x2 grid.  Tile 256 x 256 (each wave 128 x 128,
// 4 x 4 MFMA tiles, accumulators in AGPRs), or for SwiGLU 256 x 128 with two
// right operands (each wave 128 x 64 per operand).  K step 64, LDS
// double-buffered (2 x 72 KiB, rows padded to 72 elements: conflict-free
// fragment reads), global loads for the next step staged in registers during
// the current step's MFMAs.  A right operand stored [k][n] is transposed in
// registers (4 k x 8 n per thread) before the LDS write, so both operands
// read 16 contiguous bytes per lane.
//
// Epilogues: residual relation added before the store; SwiGLU stores
// silu(g) * u from its two accumulators.
#include "ea_device.h"

namespace ea {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int TM = kGemmTM;  // 256
constexpr int TK = 64;
constexpr int PITCH = TK + 8;  // LDS row pitch in elements (144 bytes)
constexpr int kThreads = 256;

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

// ---- A tile: 256 rows x 64 k, k contiguous; 2048 16-byte pieces, 8 per thread
__device__ __forceinline__ void load_a(uint4 (&r)[8], const char* base, const DevBlk& ab, int m0, int k0,
                                       int tid) {
  const int mext = ab.ext[0], kext = ab.ext[1];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int c = tid + kThreads * i;
    const int gm = m0 + (c >> 3), gk = k0 + (c & 7) * 8;
    const bool ok = gm < mext && gk < kext;
    r[i] = masked_load(base, ok ? ((int64_t)gm * kext + gk) * 2 : 0, ok);
  }
}

__device__ __forceinline__ void store_a(const uint4 (&r)[8], uint16_t* s, int tid) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int c = tid + kThreads * i;
    *reinterpret_cast<uint4*>(s + (c >> 3) * PITCH + (c & 7) * 8) = r[i];
  }
}

// ---- B tile: BN columns x 64 k, stored in LDS as [n][k]; NP 16-byte pieces
// per thread (BN = 256 -> 8, BN = 128 -> 4).
template <bool KMAJOR, int BN>
struct BTile {
  static constexpr int NP = BN * TK / 8 / kThreads;
  // [k][n] storage: blocks of 4 k x 8 n; block q = tid + 256 b, kg = q % 16, nc = q / 16
  __device__ __forceinline__ static void load(uint4 (&r)[NP], const char* base, const DevBlk& bb, int n0, int k0,
                                              int tid) {
    if constexpr (!KMAJOR) {
      const int kext = bb.ext[0], next = bb.ext[1];
#pragma unroll
      for (int b = 0; b < NP / 4; ++b) {
        const int q = tid + kThreads * b;
        const int kg = q & 15, nc = q >> 4;
        const int gn = n0 + nc * 8;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int gk = k0 + kg * 4 + i;
          const bool ok = gk < kext && gn < next;
          r[4 * b + i] = masked_load(base, ok ? ((int64_t)gk * next + gn) * 2 : 0, ok);
        }
      }
    } else {
      const int next = bb.ext[0], kext = bb.ext[1];
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
  int row0, col0;   // this lane's first row and column
};

// Accumulator r of MFMA tile (i, j) in lane l holds row 8*(r/4) + 4*(l/32) +
// r%4 and column l%32 of that 32x32 tile (row0/col0 carry the lane parts).
template <bool SWIGLU, int NB, int WN, int DT, bool RES>
__device__ __forceinline__ void epilogue(const f32x16_t (&acc)[NB][4][WN], const EpiArgs& e) {
#pragma clang loop unroll(full)
  for (int i = 0; i < 4; ++i)
#pragma clang loop unroll(full)
    for (int j = 0; j < WN; ++j)
#pragma clang loop unroll(full)
      for (int r = 0; r < 16; ++r) {
        const int gm = e.row0 + i * 32 + 8 * (r >> 2) + (r & 3);
        const int gn = e.col0 + j * 32;
        if (gm < e.mext && gn < e.next) {
          float v = acc[0][i][j][r];
          if constexpr (SWIGLU) v = v / (1.0f + __expf(-v)) * acc[NB - 1][i][j][r];
          const int64_t idx = (int64_t)gm * e.next + gn;
          if constexpr (DT == EA_F32) {
            if constexpr (RES) v += reinterpret_cast<const float*>(e.res)[idx];
            reinterpret_cast<float*>(e.c)[idx] = v;
          } else if constexpr (DT == EA_BF16) {
            if constexpr (RES) v += bf16_to_f32(reinterpret_cast<const uint16_t*>(e.res)[idx]);
            reinterpret_cast<uint16_t*>(e.c)[idx] = f32_to_bf16(v);
          } else {
            if constexpr (RES) v += f16_to_f32(reinterpret_cast<const uint16_t*>(e.res)[idx]);
            reinterpret_cast<uint16_t*>(e.c)[idx] = f32_to_f16(v);
          }
        }
      }
}

template <bool BF16, bool KMAJOR, bool SWIGLU>
__global__ __launch_bounds__(kThreads, 1) void gemm_kernel(const GemmArgs p) {
  constexpr int NB = SWIGLU ? 2 : 1;      // right operands
  constexpr int BN = SWIGLU ? 128 : 256;  // columns per right operand
  constexpr int WN = BN / 2 / 32;         // MFMA tiles per wave along n, per operand
  using BT = BTile<KMAJOR, BN>;
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][TM * PITCH];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][NB * BN * PITCH];
  __shared__ int s_last;

  // kernel arguments into registers (no address of the argument block is taken)
  const int32_t* __restrict__ tuples = p.tuples;
  const DevBlk* __restrict__ blk_a = p.blk_a;
  const DevBlk* __restrict__ blk_b = p.blk_b;
  const DevBlk* __restrict__ blk_b2 = p.blk_b2;
  const char* __restrict__ pa = p.a;
  const char* __restrict__ pb = p.b;
  const char* __restrict__ pb2 = p.b2;
  const int ts = p.tuple_stride;

  const GemmTile tile = p.tiles[blockIdx.x];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid >> 1, wn = wid & 1;
  const int g = lane >> 5, lq = lane & 31;
  const int32_t gb = p.goff[tile.block], ge = p.goff[tile.block + 1];
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

  uint4 ra[8], rb[NB][BT::NP];
  int t = t_begin, k0 = 0;
  bool have = t < t_end;
  if (have) {
    const int32_t* tp = tuples + (int64_t)t * ts;
    const DevBlk& ab = blk_a[tp[1]];
    load_a(ra, pa + ab.off, ab, tile.m0, 0, tid);
    const DevBlk& bb = blk_b[tp[2]];
    BT::load(rb[0], pb + bb.off, bb, tile.n0, 0, tid);
    if constexpr (SWIGLU) {
      const DevBlk& bb2 = blk_b2[tp[3]];
      BT::load(rb[NB - 1], pb2 + bb2.off, bb2, tile.n0, 0, tid);
    }
    store_a(ra, sA[0], tid);
#pragma unroll
    for (int o = 0; o < NB; ++o) BT::store(rb[o], sB[0] + o * BN * PITCH, tid);
  }
  __syncthreads();
  int buf = 0;
  while (have) {
    int nt = t, nk = k0 + TK;
    if (nk >= blk_a[tuples[(int64_t)t * ts + 1]].ext[1]) {
      nt = t + 1;
      nk = 0;
    }
    const bool next = nt < t_end;
    if (next) {  // prefetch the next K step into registers
      const int32_t* tp = tuples + (int64_t)nt * ts;
      const DevBlk& ab = blk_a[tp[1]];
      load_a(ra, pa + ab.off, ab, tile.m0, nk, tid);
      const DevBlk& bb = blk_b[tp[2]];
      BT::load(rb[0], pb + bb.off, bb, tile.n0, nk, tid);
      if constexpr (SWIGLU) {
        const DevBlk& bb2 = blk_b2[tp[3]];
        BT::load(rb[NB - 1], pb2 + bb2.off, bb2, tile.n0, nk, tid);
      }
    }
    const uint16_t* a_s = sA[buf] + (wm * 128 + lq) * PITCH + 8 * g;
    const uint16_t* b_s = sB[buf] + (wn * (BN / 2) + lq) * PITCH + 8 * g;
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
      __builtin_amdgcn_sched_barrier(0);  // bound the live fragment registers to one k16 step
    }
    if (next) {
      store_a(ra, sA[buf ^ 1], tid);
#pragma unroll
      for (int o = 0; o < NB; ++o) BT::store(rb[o], sB[buf ^ 1] + o * BN * PITCH, tid);
    }
    __syncthreads();
    buf ^= 1;
    t = nt;
    k0 = nk;
    have = next;
  }

  // ---- split output key: write this unit's partial sums; the last unit of
  // the key adds all partials in part order.  Partials are laid out in
  // accumulator order (lane-contiguous float4s), so the accesses coalesce.
  if (tile.n_parts > 1) {
    constexpr int PER_WAVE = NB * 4 * WN * 16;  // floats per lane
    float* mine = p.partials + ((int64_t)tile.slot * 4 + wid) * PER_WAVE * 64;
#pragma unroll
    for (int o = 0; o < NB; ++o)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4) {
            const int q = ((o * 4 + i) * WN + j) * 4 + r4;
            *reinterpret_cast<float4*>(mine + ((int64_t)q * 64 + lane) * 4) =
                make_float4(acc[o][i][j][4 * r4], acc[o][i][j][4 * r4 + 1], acc[o][i][j][4 * r4 + 2],
                            acc[o][i][j][4 * r4 + 3]);
          }
    __threadfence();
    __syncthreads();
    if (tid == 0) s_last = atomicAdd(p.counters + tile.counter, 1) == tile.n_parts - 1;
    __syncthreads();
    if (!s_last) return;
    __threadfence();
#pragma unroll
    for (int o = 0; o < NB; ++o)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j) acc[o][i][j] = f32x16_t{};
    for (int part = 0; part < tile.n_parts; ++part) {
      const float* src = p.partials + ((int64_t)(tile.first_slot + part) * 4 + wid) * PER_WAVE * 64;
#pragma unroll
      for (int o = 0; o < NB; ++o)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < WN; ++j)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
              const int q = ((o * 4 + i) * WN + j) * 4 + r4;
              const float4 v = *reinterpret_cast<const float4*>(src + ((int64_t)q * 64 + lane) * 4);
              acc[o][i][j][4 * r4] += v.x;
              acc[o][i][j][4 * r4 + 1] += v.y;
              acc[o][i][j][4 * r4 + 2] += v.z;
              acc[o][i][j][4 * r4 + 3] += v.w;
            }
    }
    if (tid == 0) p.counters[tile.counter] = 0;  // ready for the next call (stream-ordered)
  }

  // ---- epilogue (dtype and residual decided once, outside the unrolled loops)
  const DevBlk& cb = p.blk_c[tile.block];
  const EpiArgs ea_{p.c + cb.off, p.res ? p.res + cb.off : nullptr, cb.ext[0], cb.ext[1],
                    tile.m0 + wm * 128 + 4 * g, tile.n0 + wn * (BN / 2) + lq};
  if (!ea_.res && p.dt_out == EA_BF16) epilogue<SWIGLU, NB, WN, EA_BF16, false>(acc, ea_);
  else if (!ea_.res && p.dt_out == EA_F32) epilogue<SWIGLU, NB, WN, EA_F32, false>(acc, ea_);
  else if (p.dt_out == EA_BF16) epilogue<SWIGLU, NB, WN, EA_BF16, true>(acc, ea_);
  else if (p.dt_out == EA_F32) epilogue<SWIGLU, NB, WN, EA_F32, true>(acc, ea_);
  else if (!ea_.res) epilogue<SWIGLU, NB, WN, EA_F16, false>(acc, ea_);
  else epilogue<SWIGLU, NB, WN, EA_F16, true>(acc, ea_);
}

template <bool BF16, bool KMAJOR, bool SWIGLU>
hipError_t launch3(const GemmArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((gemm_kernel<BF16, KMAJOR, SWIGLU>), dim3((uint32_t)a.n_tiles), dim3(kThreads), 0, s, a);
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

}  // namespace

hipError_t launch_gemm(const GemmArgs& a, hipStream_t s) {
  if (a.n_tiles == 0) return hipSuccess;
  return a.dt_in == EA_BF16 ? launch1<true>(a, s) : launch1<false>(a, s);
}

}  // namespace ea
