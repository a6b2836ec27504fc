// ea_gemm32.hip -- fp32 block-product join-agg ("ab,bc->ac" or "ab,cb->ac"
// over f32 relations) on the vector ALUs.
//
// Section 3.2, Example "Matrix multiply, decomposed": every tuple of an
// output key multiplies one block of A by one block of B and the products
// are summed (aggregation +).  A workgroup owns a 32 x 32 tile of one output
// block and walks the key's tuples in order, so the SUM over the key's blocks
// stays in registers and the result is stored once.  Per tuple, the
// contracted extent is taken 64 at a time: a 32 x 64 slice of A and a 64 x 32
// slice of B are staged in LDS (masked at block edges), the next slices being
// loaded into registers meanwhile, and each of the 256 threads accumulates a
// 2 x 2 patch of the tile with fp32 FMAs, in ascending contracted order
// (deterministic).
#include "ea_device.h"

namespace ea {

namespace {

constexpr int kT = kGemm32Tile;  // output tile (32 x 32)
constexpr int kK = 64;           // contracted slice per LDS stage
constexpr int kThreads = 256;
constexpr int kPer = kT * kK / kThreads;  // elements of each operand slice per thread (8)

__global__ __launch_bounds__(kThreads) void gemm32_kernel(const Gemm32Args p) {
  __shared__ float sA[kT][kK + 1];  // [m][k], padded against bank conflicts
  __shared__ float sB[kK][kT + 1];  // [k][n]
  const Gemm32Work w = p.work[blockIdx.x];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;  // 2 x 2 outputs per thread
  const int32_t gb = p.goff[w.block], ge = p.goff[w.block + 1];
  const DevBlk& cb = p.blk_c[w.block];
  const int mext = cb.ext[0], next = cb.ext[1];
  // the walk over the key's tuples, kK of the contracted extent per step;
  // the next step's slices are loaded into registers while this one is
  // computed from the LDS
  float ra[kPer], rb[kPer];
  auto load = [&](int t, int k0) {
    const int32_t* tp = p.tuples + (int64_t)t * p.tuple_stride;
    const DevBlk& ab = p.blk_a[tp[1]];
    const DevBlk& bb = p.blk_b[tp[2]];
    const float* A = reinterpret_cast<const float*>(p.a + ab.off);
    const float* B = reinterpret_cast<const float*>(p.b + bb.off);
    const int am = ab.ext[0], ak = ab.ext[1];
    const int bn = p.b_kmajor ? bb.ext[0] : bb.ext[1];  // B is [k][n], or [n][k] when b_kmajor
#pragma unroll
    for (int r = 0; r < kPer; ++r) {
      const int e = tid + kThreads * r;
      const int m = e / kK, k = e % kK;  // consecutive threads along k of a row of A
      const int gm = w.m0 + m, gk = k0 + k;
      ra[r] = gm < am && gk < ak ? A[(int64_t)gm * ak + gk] : 0.0f;
      int kb, n;
      if (p.b_kmajor) {  // consecutive threads along k of a row of B[n][k]
        n = e / kK;
        kb = e % kK;
      } else {           // consecutive threads along n of a row of B[k][n]
        kb = e / kT;
        n = e % kT;
      }
      const int gn = w.n0 + n, gkb = k0 + kb;
      rb[r] = gn < bn && gkb < ak ? (p.b_kmajor ? B[(int64_t)gn * ak + gkb] : B[(int64_t)gkb * bn + gn]) : 0.0f;
    }
  };
  auto stash = [&]() {
#pragma unroll
    for (int r = 0; r < kPer; ++r) {
      const int e = tid + kThreads * r;
      sA[e / kK][e % kK] = ra[r];
      if (p.b_kmajor) sB[e % kK][e / kK] = rb[r];
      else sB[e / kT][e % kT] = rb[r];
    }
  };
  auto extent = [&](int t) { return p.blk_a[p.tuples[(int64_t)t * p.tuple_stride + 1]].ext[1]; };
  float acc[2][2] = {{0.0f, 0.0f}, {0.0f, 0.0f}};
  int t = gb, k0 = 0;
  while (t < ge && extent(t) == 0) ++t;
  if (t < ge) load(t, k0);
  while (t < ge) {
    stash();
    __syncthreads();
    // the next step (if any) goes out before this one is computed
    int nt = t, nk = k0 + kK;
    if (nk >= extent(nt)) {
      ++nt;
      nk = 0;
      while (nt < ge && extent(nt) == 0) ++nt;
    }
    if (nt < ge) load(nt, nk);
#pragma unroll 16
    for (int k = 0; k < kK; ++k) {
      const float a0 = sA[ty * 2][k], a1 = sA[ty * 2 + 1][k];
      const float b0 = sB[k][tx * 2], b1 = sB[k][tx * 2 + 1];
      acc[0][0] = fmaf(a0, b0, acc[0][0]);
      acc[0][1] = fmaf(a0, b1, acc[0][1]);
      acc[1][0] = fmaf(a1, b0, acc[1][0]);
      acc[1][1] = fmaf(a1, b1, acc[1][1]);
    }
    __syncthreads();
    t = nt;
    k0 = nk;
  }
  char* C = p.c + cb.off;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int gm = w.m0 + ty * 2 + i;
    if (gm >= mext) continue;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int gn = w.n0 + tx * 2 + j;
      if (gn >= next) continue;
      const int64_t idx = (int64_t)gm * next + gn;
      if (p.dt_out == EA_F32) reinterpret_cast<float*>(C)[idx] = acc[i][j];
      else if (p.dt_out == EA_BF16) reinterpret_cast<uint16_t*>(C)[idx] = f32_to_bf16(acc[i][j]);
      else reinterpret_cast<uint16_t*>(C)[idx] = f32_to_f16(acc[i][j]);
    }
  }
}

}  // namespace

hipError_t launch_gemm32(const Gemm32Args& a, hipStream_t s) {
  if (a.n_work == 0) return hipSuccess;
  hipLaunchKernelGGL(gemm32_kernel, dim3((uint32_t)a.n_work), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace ea
