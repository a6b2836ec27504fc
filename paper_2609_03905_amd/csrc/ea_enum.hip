// ea_enum.hip -- the join enumerator (Section 3.2, Definition "Implementation",
// step 1; Section 3.3 for the product-of-intervals count).
//
// One workgroup walks the letter-block space in canonical order (group
// letters first, then the remaining letters in order of first appearance,
// last letter fastest).  Each candidate is matched against every operand's
// block keys: for each of the operand's letters the candidate interval
// (lo, hi) must be one of the operand's intervals (binary search on its split
// points, then an exact comparison of both bounds).  A matched candidate that
// passes the optional predicates (causal; grouped-query heads; packed
// sequences, Section 3.3 Example "Flash attention") becomes a tuple
// (output block, input blocks...).  Kept tuples are compacted with a
// workgroup prefix sum, so the table comes out grouped by output key with no
// sort, and the CSR group offsets fall out of the same scan.
#include "ea_device.h"

namespace ea {

namespace {

constexpr int kThreads = 1024;

__device__ __forceinline__ int find_interval(const int32_t* s, int n, int32_t lo, int32_t hi) {
  int a = 0, z = n;  // invariant: s[a] <= lo < s[z] (s[n] is the extent)
  if (lo < s[0] || lo >= s[n]) return -1;
  while (z - a > 1) {
    const int m = (a + z) >> 1;
    if (s[m] <= lo) a = m;
    else z = m;
  }
  return (s[a] == lo && s[a + 1] == hi) ? a : -1;
}

// index of the sequence holding position x: the first end above it
__device__ __forceinline__ int seq_of(const int32_t* ends, int n, int32_t x) {
  int a = 0, z = n;  // invariant: every end before a is <= x, end z-1 (if z < n) is > x
  while (a < z) {
    const int m = (a + z) >> 1;
    if (ends[m] <= x) a = m + 1;
    else z = m;
  }
  return a;
}

__global__ __launch_bounds__(kThreads) void enumerate_kernel(const EnumDesc* __restrict__ dp,
                                                             const int32_t* __restrict__ splits,
                                                             int32_t* __restrict__ tuples,
                                                             int32_t* __restrict__ goff,
                                                             int32_t* __restrict__ count) {
  __shared__ EnumDesc d;
  __shared__ int32_t wave_sums[kThreads / 64];
  {
    const int32_t* src = reinterpret_cast<const int32_t*>(dp);
    int32_t* dst = reinterpret_cast<int32_t*>(&d);
    for (int i = threadIdx.x; i < (int)(sizeof(EnumDesc) / 4); i += kThreads) dst[i] = src[i];
  }
  __syncthreads();
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int stride = d.n_in + 1;
  int32_t total = 0;
  for (int64_t c0 = 0; c0 < d.n_cand; c0 += kThreads) {
    const int64_t c = c0 + tid;
    bool keep = false;
    int32_t rec[kMaxOps];
    if (c < d.n_cand) {
      int32_t coord[kMaxLetters];
      int64_t rem = c;
      for (int l = d.n_letters - 1; l >= 0; --l) {
        coord[l] = (int32_t)(rem % d.letter_nb[l]);
        rem /= d.letter_nb[l];
      }
      keep = true;
      for (int o = 0; o <= d.n_in && keep; ++o) {
        int32_t b = 0;
        for (int dd = 0; dd < d.op_rank[o]; ++dd) {
          const int L = d.op_letter[o][dd];
          const int32_t lo = splits[d.letter_split[L] + coord[L]];
          const int32_t hi = splits[d.letter_split[L] + coord[L] + 1];
          const int n = d.op_nb[o][dd];
          const int a = find_interval(splits + d.op_split[o][dd], n, lo, hi);
          if (a < 0) {
            keep = false;
            break;
          }
          b = b * n + a;
        }
        rec[o == d.n_in ? 0 : o + 1] = b;
      }
      if (keep && d.causal) {
        const int32_t q_hi = splits[d.letter_split[d.cq] + coord[d.cq] + 1];
        const int32_t k_lo = splits[d.letter_split[d.ck] + coord[d.ck]];
        keep = k_lo <= q_hi - 1;
      }
      if (keep && d.gqa > 1) {  // the K/V head block holds the Q head block's heads / gqa
        const int32_t h_lo = splits[d.letter_split[d.gh] + coord[d.gh]];
        const int32_t h_hi = splits[d.letter_split[d.gh] + coord[d.gh] + 1];
        const int32_t g_lo = splits[d.letter_split[d.gg] + coord[d.gg]];
        const int32_t g_hi = splits[d.letter_split[d.gg] + coord[d.gg] + 1];
        keep = (int64_t)g_lo * d.gqa <= h_lo && h_hi <= (int64_t)g_hi * d.gqa;
      }
      if (keep && d.n_seq > 0) {  // query and key blocks in one sequence (no block straddles one)
        const int32_t q_lo = splits[d.letter_split[d.cq] + coord[d.cq]];
        const int32_t k_lo = splits[d.letter_split[d.ck] + coord[d.ck]];
        keep = seq_of(splits + d.seq_split, d.n_seq, q_lo) == seq_of(splits + d.seq_split, d.n_seq, k_lo);
      }
    }
    const uint64_t mask = __ballot(keep);
    const int pre = __popcll(mask & ((1ull << lane) - 1ull));
    if (lane == 0) wave_sums[wid] = __popcll(mask);
    __syncthreads();
    int wbase = 0, ctotal = 0;
    for (int w = 0; w < kThreads / 64; ++w) {
      wbase += w < wid ? wave_sums[w] : 0;
      ctotal += wave_sums[w];
    }
    const int32_t pos = total + wbase + pre;
    if (keep)
      for (int o = 0; o < stride; ++o) tuples[(int64_t)pos * stride + o] = rec[o];
    if (c < d.n_cand && c % d.per_group == 0) goff[c / d.per_group] = pos;
    total += ctotal;
    __syncthreads();
  }
  if (tid == 0) {
    goff[d.n_groups] = total;
    *count = total;
  }
}

}  // namespace

hipError_t launch_enumerate(const EnumDesc* d_desc, const int32_t* d_splits, int32_t* d_tuples, int32_t* d_goff,
                            int32_t* d_count, hipStream_t s) {
  hipLaunchKernelGGL(enumerate_kernel, dim3(1), dim3(kThreads), 0, s, d_desc, d_splits, d_tuples, d_goff,
                     d_count);
  return hipGetLastError();
}

}  // namespace ea
