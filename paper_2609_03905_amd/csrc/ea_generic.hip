// ea_generic.hip -- the general einsum join-agg (Section 3.2, Definition
// "Implementation"): any spec, join MUL or ADD, aggregation NONE, SUM or MAX.
//
// One thread owns one element of one output block.  It walks its group's
// tuples in table order and, inside each tuple, every value of the contracted
// letters within the tuple blocks' intervals, applying the join to the
// inputs' elements and the aggregation to the running value in f32.  This is
// the slow, general path; two-operand bf16/f16 products take the matrix-core
// kernel instead.
#include "ea_device.h"

namespace ea {

namespace {

__global__ __launch_bounds__(256) void generic_kernel(GenArgs a) {
  const GenDesc& g = *a.desc;
  const GenWork w = a.work[blockIdx.x];
  const DevBlk& ob = a.blk[g.n_in][w.block];
  int64_t n = 1;
  for (int d = 0; d < g.out_rank; ++d) n *= ob.ext[d];
  const int64_t e = (int64_t)w.start + threadIdx.x;
  if (e >= n) return;
  int32_t val[kMaxLetters];
  {
    int64_t rem = e;
    for (int d = g.out_rank - 1; d >= 0; --d) {
      val[g.out_letter[d]] = ob.lo[d] + (int32_t)(rem % ob.ext[d]);
      rem /= ob.ext[d];
    }
  }
  float acc = g.agg == EA_AGG_MAX ? -INFINITY : 0.0f;
  const int stride = g.n_in + 1;
  const int32_t t0 = a.goff[w.block], t1 = a.goff[w.block + 1];
  for (int32_t t = t0; t < t1; ++t) {
    const int32_t* tp = a.tuples + (int64_t)t * stride;
    int32_t clo[kMaxLetters], cext[kMaxLetters];
    int64_t ncomb = 1;
    for (int j = 0; j < g.n_contr; ++j) {
      const DevBlk& b = a.blk[g.contr_op[j]][tp[1 + g.contr_op[j]]];
      clo[j] = b.lo[g.contr_dim[j]];
      cext[j] = b.ext[g.contr_dim[j]];
      ncomb *= cext[j];
    }
    for (int64_t cc = 0; cc < ncomb; ++cc) {
      int64_t rem = cc;
      for (int j = g.n_contr - 1; j >= 0; --j) {
        val[g.contr_letter[j]] = clo[j] + (int32_t)(rem % cext[j]);
        rem /= cext[j];
      }
      float f = g.join == EA_JOIN_MUL ? 1.0f : 0.0f;
      for (int i = 0; i < g.n_in; ++i) {
        const DevBlk& b = a.blk[i][tp[1 + i]];
        int64_t idx = 0;
        for (int d = 0; d < g.in_rank[i]; ++d) idx = idx * b.ext[d] + (val[g.in_letter[i][d]] - b.lo[d]);
        const float x = ld_elem(a.in[i] + b.off, idx, g.dt_in[i]);
        f = g.join == EA_JOIN_MUL ? f * x : f + x;
      }
      if (g.agg == EA_AGG_MAX) acc = fmaxf(acc, f);
      else if (g.agg == EA_AGG_SUM) acc += f;
      else acc = f;
    }
  }
  if (g.has_res) acc += ld_elem(a.res + ob.off, e, g.dt_res);
  st_elem(a.out + ob.off, e, g.dt_out, acc);
}

}  // namespace

hipError_t launch_generic(const GenArgs& a, hipStream_t s) {
  if (a.n_work == 0) return hipSuccess;
  hipLaunchKernelGGL(generic_kernel, dim3((uint32_t)a.n_work), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace ea
