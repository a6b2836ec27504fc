// ea_repart.hip -- local repartition (Section 5.3: the overlay of the source
// and destination partitions gives atoms; decompose slices source blocks into
// atoms, recompose concatenates atoms into destination blocks).
//
// Both steps are fused into one pass of vector copies: the host cuts the
// tensor into boxes (source block intersected with destination block, each a
// union of overlay atoms) and each workgroup copies a byte range of one box,
// 16 bytes per lane where alignment allows.  Pure data movement: bit-exact.
#include "ea_device.h"

namespace ea {

namespace {

template <int VEC>
struct Vec;
template <>
struct Vec<16> { using T = uint4; };
template <>
struct Vec<8> { using T = uint2; };
template <>
struct Vec<4> { using T = uint32_t; };
template <>
struct Vec<2> { using T = uint16_t; };
template <>
struct Vec<1> { using T = uint8_t; };

constexpr int kThreads = 256;

// Byte offsets (source, destination) of byte L of the task's box.  Rows of a
// power-of-two width take a shift instead of a division, and a box with one
// outer dim (the usual 2-d block) needs no further division.
__device__ __forceinline__ void box_offsets(const RepTask& t, int32_t L, int64_t& so, int64_t& dof) {
  const int sh = t.row_shift;
  int32_t row = sh >= 0 ? L >> sh : L / t.row_bytes;
  const int32_t col = L - row * t.row_bytes;
  so = col;
  dof = col;
  if (t.n_outer == 1) {  // row < outer_ext[0] for every byte of the range
    so += (int64_t)row * t.src_stride[0];
    dof += (int64_t)row * t.dst_stride[0];
    return;
  }
  for (int d = t.n_outer - 1; d >= 0; --d) {
    const int32_t c = row % t.outer_ext[d];
    row /= t.outer_ext[d];
    so += (int64_t)c * t.src_stride[d];
    dof += (int64_t)c * t.dst_stride[d];
  }
}

// UNROLL vectors per thread are loaded before any is stored: 4 for tasks of
// kRepTaskBytes, 2 for tasks of kRepTaskBytesSmall (one pass of the workgroup
// for 16-byte vectors).
template <int VEC, bool STREAM, int UNROLL>
__device__ __forceinline__ void copy_range(const RepTask* __restrict__ tp, const char* __restrict__ src,
                                           char* __restrict__ dst) {
  using T = typename Vec<VEC>::T;
  const RepTask& t = *tp;  // fields read from global memory, never copied to the stack
  const char* s0 = src + t.src_off;
  char* d0 = dst + t.dst_off;
  const int32_t end = t.end;
  // UNROLL loads in flight per thread, then their stores.  A vector past the
  // range is redirected to the range's first vector: it loads that vector and
  // stores it to its own destination again (the same bytes that lane 0
  // writes), so neither loads nor stores carry a condition and all the loads
  // are issued before the first store.
  for (int32_t L0 = t.begin + threadIdx.x * VEC; L0 < end; L0 += kThreads * VEC * UNROLL) {
    int64_t sos[UNROLL], dofs[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const int32_t L = L0 + u * kThreads * VEC;
      box_offsets(t, L < end ? L : t.begin, sos[u], dofs[u]);
    }
    T v[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) v[u] = *reinterpret_cast<const T*>(s0 + sos[u]);
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) store_out<STREAM>(d0 + dofs[u], v[u]);
  }
}

template <bool STREAM, int UNROLL>
__global__ __launch_bounds__(kThreads) void repart_kernel(const RepTask* __restrict__ tasks,
                                                          const char* __restrict__ src, char* __restrict__ dst) {
  const RepTask* t = tasks + blockIdx.x;
  switch (t->vec) {
    case 16: copy_range<16, STREAM, UNROLL>(t, src, dst); break;
    case 8: copy_range<8, STREAM, UNROLL>(t, src, dst); break;
    case 4: copy_range<4, STREAM, UNROLL>(t, src, dst); break;
    case 2: copy_range<2, STREAM, UNROLL>(t, src, dst); break;
    default: copy_range<1, STREAM, UNROLL>(t, src, dst); break;
  }
}
static_assert(kRepTaskBytes == kThreads * 4 * 16 && kRepTaskBytesSmall == kThreads * 2 * 16, "task sizes");

}  // namespace

hipError_t launch_repartition(const RepTask* d_tasks, int64_t n_tasks, const char* src, char* dst, bool stream_out,
                              bool small_tasks, hipStream_t s) {
  if (n_tasks == 0) return hipSuccess;
  const dim3 grid((uint32_t)n_tasks), block(kThreads);
  if (small_tasks) {
    if (stream_out) hipLaunchKernelGGL((repart_kernel<true, 2>), grid, block, 0, s, d_tasks, src, dst);
    else hipLaunchKernelGGL((repart_kernel<false, 2>), grid, block, 0, s, d_tasks, src, dst);
  } else {
    if (stream_out) hipLaunchKernelGGL((repart_kernel<true, 4>), grid, block, 0, s, d_tasks, src, dst);
    else hipLaunchKernelGGL((repart_kernel<false, 4>), grid, block, 0, s, d_tasks, src, dst);
  }
  return hipGetLastError();
}

}  // namespace ea
