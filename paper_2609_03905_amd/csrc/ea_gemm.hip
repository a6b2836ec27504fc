// ea_gemm.hip -- block-GEMM join-agg on the CDNA4 matrix cores.
//
// Section 3.2, Example "Matrix multiply, decomposed": the per-tuple concrete
// operator is a block matrix product and the aggregation is +.  Here one
// workgroup owns a 128x128 tile of one output block (one output key) and
// runs the K-loop across *all tuples of that key's group*, so the SUM of the
// partial products happens in the MFMA accumulators and no partial block ever
// reaches memory; the recompose step is the store into the output block.
//
// Inputs bf16 or f16, fp32 accumulation (v_mfma_f32_32x32x16_{bf16,f16}).
// Tile: 256 threads = 4 waves in a 2x2 grid, each wave 64x64 = 2x2 MFMA
// tiles; K step 64.  Operands are staged through LDS (double-buffered, rows
// padded to 72 elements so the MFMA fragment reads of 32 consecutive rows hit
// distinct banks).  A right operand stored [k][n] is transposed in registers
// (4 rows x 8 columns per thread) before it is written to LDS as [n][k], so
// both MFMA operands read 16 contiguous bytes per lane.
//
// Epilogues: optional residual relation added before the store; SwiGLU
// computes two products from one A stream and stores silu(g) * u.
#include "ea_device.h"

namespace ea {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int TM = kGemmTM, TN = kGemmTN, TK = 64;
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

// 16-byte load that yields zeros when !ok.  The load itself always happens at
// an in-bounds address (the block base when masked; every block row holds at
// least 16 bytes on this path), so no branch or pointer select is needed.
__device__ __forceinline__ uint4 masked_load(const char* base, int64_t off, bool ok) {
  const uint4 v = *reinterpret_cast<const uint4*>(base + off);
  return ok ? v : make_uint4(0, 0, 0, 0);
}

__device__ __forceinline__ uint32_t word(const uint4& v, int w) {
  return w == 0 ? v.x : w == 1 ? v.y : w == 2 ? v.z : v.w;
}

template <bool KMAJOR>
struct BLoader {
  // [k][n] storage: thread covers rows k = 4*kg .. 4*kg+3, columns 8*nc .. 8*nc+7.
  // [n][k] storage: like A, chunk c = tid + 256*i -> row n = c/8, k chunk c%8.
  __device__ __forceinline__ static void load(uint4 (&r)[4], const char* base, const DevBlk& bb, int n0, int k0,
                                              int tid) {
    if constexpr (!KMAJOR) {
      const int kext = bb.ext[0], next = bb.ext[1];
      const int kg = tid & 15, nc = tid >> 4;
      const int gn = n0 + nc * 8;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int gk = k0 + kg * 4 + i;
        const bool ok = gk < kext && gn < next;
        r[i] = masked_load(base, ok ? ((int64_t)gk * next + gn) * 2 : 0, ok);
      }
    } else {
      const int next = bb.ext[0], kext = bb.ext[1];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = tid + kThreads * i;
        const int gn = n0 + (c >> 3), gk = k0 + (c & 7) * 8;
        const bool ok = gn < next && gk < kext;
        r[i] = masked_load(base, ok ? ((int64_t)gn * kext + gk) * 2 : 0, ok);
      }
    }
  }
  __device__ __forceinline__ static void store(const uint4 (&r)[4], uint16_t* s, int tid) {
    if constexpr (!KMAJOR) {
      const int kg = tid & 15, nc = tid >> 4;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int w = j >> 1;
        const uint32_t x0 = word(r[0], w), x1 = word(r[1], w), x2 = word(r[2], w), x3 = word(r[3], w);
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
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = tid + kThreads * i;
        *reinterpret_cast<uint4*>(s + (c >> 3) * PITCH + (c & 7) * 8) = r[i];
      }
    }
  }
};

__device__ __forceinline__ void load_a(uint4 (&r)[4], const char* base, const DevBlk& ab, int m0, int k0,
                                       int tid) {
  const int mext = ab.ext[0], kext = ab.ext[1];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + kThreads * i;
    const int gm = m0 + (c >> 3), gk = k0 + (c & 7) * 8;
    const bool ok = gm < mext && gk < kext;
    r[i] = masked_load(base, ok ? ((int64_t)gm * kext + gk) * 2 : 0, ok);
  }
}

__device__ __forceinline__ void store_a(const uint4 (&r)[4], uint16_t* s, int tid) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + kThreads * i;
    *reinterpret_cast<uint4*>(s + (c >> 3) * PITCH + (c & 7) * 8) = r[i];
  }
}

template <bool BF16, bool KMAJOR, bool SWIGLU>
__global__ __launch_bounds__(kThreads) void gemm_kernel(const GemmArgs p) {
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][TM * PITCH];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][TN * PITCH];
  __shared__ __attribute__((aligned(16))) uint16_t sB2[SWIGLU ? 2 : 1][SWIGLU ? TN * PITCH : 8];

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
  const int32_t t0 = p.goff[tile.block], t1 = p.goff[tile.block + 1];

  f32x16_t acc[2][2], acc2[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      acc[i][j] = f32x16_t{};
      acc2[i][j] = f32x16_t{};
    }

  uint4 ra[4], rb[4], rb2[4];
  int t = t0, k0 = 0;
  bool have = t < t1;
  if (have) {
    const int32_t* tp = tuples + (int64_t)t * ts;
    const DevBlk& ab = blk_a[tp[1]];
    load_a(ra, pa + ab.off, ab, tile.m0, 0, tid);
    const DevBlk& bb = blk_b[tp[2]];
    BLoader<KMAJOR>::load(rb, pb + bb.off, bb, tile.n0, 0, tid);
    if constexpr (SWIGLU) {
      const DevBlk& bb2 = blk_b2[tp[3]];
      BLoader<KMAJOR>::load(rb2, pb2 + bb2.off, bb2, tile.n0, 0, tid);
    }
    store_a(ra, sA[0], tid);
    BLoader<KMAJOR>::store(rb, sB[0], tid);
    if constexpr (SWIGLU) BLoader<KMAJOR>::store(rb2, sB2[0], tid);
  }
  __syncthreads();
  int buf = 0;
  const int frag_k = 8 * (lane >> 5);
  while (have) {
    int nt = t, nk = k0 + TK;
    if (nk >= blk_a[tuples[(int64_t)t * ts + 1]].ext[1]) {
      nt = t + 1;
      nk = 0;
    }
    const bool next = nt < t1;
    if (next) {  // prefetch the next K step into registers
      const int32_t* tp = tuples + (int64_t)nt * ts;
      const DevBlk& ab = blk_a[tp[1]];
      load_a(ra, pa + ab.off, ab, tile.m0, nk, tid);
      const DevBlk& bb = blk_b[tp[2]];
      BLoader<KMAJOR>::load(rb, pb + bb.off, bb, tile.n0, nk, tid);
      if constexpr (SWIGLU) {
        const DevBlk& bb2 = blk_b2[tp[3]];
        BLoader<KMAJOR>::load(rb2, pb2 + bb2.off, bb2, tile.n0, nk, tid);
      }
    }
    const uint16_t* a_s = sA[buf];
    const uint16_t* b_s = sB[buf];
#pragma unroll
    for (int s = 0; s < TK / 16; ++s) {
      uint4 af[2], bf[2], bf2[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        af[i] = *reinterpret_cast<const uint4*>(a_s + (wm * 64 + i * 32 + (lane & 31)) * PITCH + s * 16 + frag_k);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        bf[j] = *reinterpret_cast<const uint4*>(b_s + (wn * 64 + j * 32 + (lane & 31)) * PITCH + s * 16 + frag_k);
      if constexpr (SWIGLU) {
#pragma unroll
        for (int j = 0; j < 2; ++j)
          bf2[j] = *reinterpret_cast<const uint4*>(sB2[buf] + (wn * 64 + j * 32 + (lane & 31)) * PITCH + s * 16 +
                                                   frag_k);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          acc[i][j] = mfma<BF16>(af[i], bf[j], acc[i][j]);
          if constexpr (SWIGLU) acc2[i][j] = mfma<BF16>(af[i], bf2[j], acc2[i][j]);
        }
    }
    if (next) {
      store_a(ra, sA[buf ^ 1], tid);
      BLoader<KMAJOR>::store(rb, sB[buf ^ 1], tid);
      if constexpr (SWIGLU) BLoader<KMAJOR>::store(rb2, sB2[buf ^ 1], tid);
    }
    __syncthreads();
    buf ^= 1;
    t = nt;
    k0 = nk;
    have = next;
  }

  // Epilogue.  Accumulator r of MFMA tile (i, j) in lane l holds row
  // 8*(r/4) + 4*(l/32) + r%4 and column l%32 of that 32x32 tile.
  const DevBlk& cb = p.blk_c[tile.block];
  const int mext = cb.ext[0], next_c = cb.ext[1];
  char* cbase = p.c + cb.off;
  const char* rbase = p.res ? p.res + cb.off : nullptr;
  const int dt_res = p.dt_res, dt_out = p.dt_out;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int gm = tile.m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int gn = tile.n0 + wn * 64 + j * 32 + (lane & 31);
        if (gm < mext && gn < next_c) {
          float v = acc[i][j][r];
          if constexpr (SWIGLU) v = v / (1.0f + __expf(-v)) * acc2[i][j][r];
          const int64_t idx = (int64_t)gm * next_c + gn;
          if (rbase) v += ld_elem(rbase, idx, dt_res);
          st_elem(cbase, idx, dt_out, v);
        }
      }
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
