// ea_rows.hip -- row-reduction join-aggs: RMSNorm and softmax.
//
// The normalised letter (the last one) is split into blocks, so a row is the
// concatenation of one segment per tuple of its group (Section 3.2,
// Definition "Implementation": the per-tuple partials -- a sum of squares, or
// a max and a sum of exponentials -- are aggregated across the group's
// blocks).  One wavefront owns one row: it loads every segment of the row
// into registers (16-byte vector loads, lanes interleaved across the row),
// forms its local partials, aggregates them across lanes (the aggregation
// across blocks, in a fixed order), and writes the normalised row from the
// registers.  HBM traffic: one read of the visible inputs, one write.
// Long bf16 RMSNorm rows (more than 512 chunks) on the affine layout are
// shared by two wavefronts, whose partial sums of squares meet in LDS.
//
// Causal softmax skips the loads of keys after the row's query position and
// stores zeros there.  Rows too long for registers, or segments that are not
// 16-byte multiples, take a scalar path that re-reads the row.
#include <type_traits>

#include "ea_device.h"

namespace ea {

namespace {

constexpr int kThreads = 64 * kRowsPerTask;  // one row per wavefront
constexpr int kMaxSeg = 64;    // segments per row on the register path
constexpr int kMaxK = 16;      // 16-byte chunks per lane on the register path

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

struct SegTable {
  int32_t start[kMaxSeg];  // first chunk of the segment within the row
  int64_t xoff[kMaxSeg];   // byte offset of the row's segment in x
  int64_t yoff[kMaxSeg];   // element index base in y's block (by offset)
  int64_t woff[kMaxSeg];   // byte offset of the w block (RMSNorm)
  int32_t klo[kMaxSeg];    // position of the segment's first element
  int32_t len[kMaxSeg];    // elements in the segment
};

struct RowInfo {
  int32_t t0, nseg;
  int32_t row;     // row index inside the group's blocks
  int32_t qpos;    // query position of the row (softmax causal)
};

__device__ __forceinline__ RowInfo row_info(const RowArgs& a, int task_row) {
  const RowTask& task = a.tasks[blockIdx.x];
  RowInfo ri;
  const int g = task.g;
  ri.row = task.row0 + task_row;
  ri.t0 = a.goff[g];
  ri.nseg = a.goff[g + 1] - ri.t0;
  ri.qpos = 0;
  if (a.causal && ri.nseg > 0) {
    const DevBlk& xb = a.blk_x[a.tuples[(int64_t)ri.t0 * a.tuple_stride + 1]];
    const int qd = a.rank - 2;
    ri.qpos = xb.lo[qd] + ri.row % xb.ext[qd];
  }
  return ri;
}

// Fill the wave's segment table (lane s describes segment s).  Returns the
// row's total chunk count.
__device__ __forceinline__ int fill_segments(const RowArgs& a, const RowInfo& ri, SegTable& st, int lane,
                                             int es) {
  const int d_last = a.rank - 1;
  int chunks = 0;
  if (lane < ri.nseg) {
    const int32_t* tp = a.tuples + (int64_t)(ri.t0 + lane) * a.tuple_stride;
    const DevBlk& xb = a.blk_x[tp[1]];
    const DevBlk& yb = a.blk_y[tp[0]];
    const int L = xb.ext[d_last];
    chunks = L * es / 16;
    st.xoff[lane] = xb.off + (int64_t)ri.row * L * es;
    st.yoff[lane] = yb.off;
    st.woff[lane] = a.blk_w ? a.blk_w[tp[2]].off : 0;
    st.klo[lane] = xb.lo[d_last];
    st.len[lane] = L;
  }
  // exclusive prefix sum of chunk counts across lanes
  int incl = chunks;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(incl, o, 64);
    if (lane >= o) incl += v;
  }
  if (lane < ri.nseg) st.start[lane] = incl - chunks;
  return __shfl(incl, 63, 64);
}

__device__ __forceinline__ int seg_of(const SegTable& st, int nseg, int chunk) {
  int s = 0;
  for (int j = 1; j < nseg; ++j) s = chunk >= st.start[j] ? j : s;
  return s;
}

template <typename T>
__device__ __forceinline__ void unpack(const uint4& v, float (&f)[8]);

template <>
__device__ __forceinline__ void unpack<uint16_t>(const uint4& v, float (&f)[8]) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

template <>
__device__ __forceinline__ void unpack<float>(const uint4& v, float (&f)[8]) {
  f[0] = __uint_as_float(v.x);
  f[1] = __uint_as_float(v.y);
  f[2] = __uint_as_float(v.z);
  f[3] = __uint_as_float(v.w);
}

// ---------------------------------------------------------------------------
// register path; XT: uint16_t for bf16 rows, float for f32 rows
// ---------------------------------------------------------------------------
// K: 16-byte chunks of the row per lane (4, 8 or 16), chosen from the row
// length so that short rows keep few registers and many waves per SIMD.
// AFF: affine layout (RowArgs::affine): addresses come from the task record
// and the strides, so the row loads go out at once; otherwise each wave
// first builds its row's segment table from the join's tuples.
// WPR: wavefronts per row.  2 halves the registers and the serial work of a
// long row (RMSNorm on the affine layout with bf16 weights only): each wave
// takes K chunks of its half, and the two partial sums of squares meet in LDS.
template <typename XT, bool SOFTMAX, int K, bool AFF, int WPR = 1>
__global__ __launch_bounds__(kThreads * WPR) void rows_vec_kernel(RowArgs a) {
  static_assert(WPR == 1 || (WPR == 2 && !SOFTMAX && AFF && sizeof(XT) == 2), "split rows: bf16 RMSNorm, affine");
  __shared__ SegTable tabs[AFF ? 1 : kThreads / 64];
  __shared__ float s_half[WPR == 2 ? kRowsPerTask * 2 : 1];
  // RMSNorm: the weights of the group's row, in the row's chunk order as
  // fp32 (EPC values per chunk), staged once for the workgroup's rows
  constexpr int ES = sizeof(XT), EPC = 16 / ES;
  __shared__ float sw[SOFTMAX ? 1 : K * WPR * 64 * EPC];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int wrow = wid / WPR;                   // the wave's row of the task
  const int cbase = (wid % WPR) * K * 64;       // first chunk of the wave's part of the row
  const RowTask& task = a.tasks[blockIdx.x];
  const bool active = wrow < ld_uniform(&task.nrows);  // waves past the task's rows only help stage the weights
  const int esy = a.dt_y == EA_F32 ? 4 : 2;
  SegTable& st = tabs[AFF ? 0 : wid];
  int total, nseg;
  int qpos = 0;
  int64_t xrow = 0, yrow = 0;
  RowInfo ri{};
  if constexpr (AFF) {
    nseg = a.nseg;
    total = nseg * a.seg_chunks;
    const int row = ld_uniform(&task.row0) + wrow;
    xrow = ld_uniform(&task.xrow) + (int64_t)wrow * a.seg_len * ES;
    yrow = ld_uniform(&task.yrow) + (int64_t)wrow * a.seg_len * esy;
    if (SOFTMAX && a.causal) qpos = ld_uniform(&task.qlo) + row % ld_uniform(&task.qext);
  } else {
    ri = row_info(a, wid);  // every row of the task is in the same group
    total = fill_segments(a, ri, st, lane, ES);
    nseg = ri.nseg;
    qpos = ri.qpos;
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }

  // Segment of a chunk: direct when every segment but the last has the same
  // chunk count (the usual even split, ragged tail allowed), else a scan of
  // the segment table.
  const int cps = a.seg_chunks;
  // chunk index -> segment, c / cps: floor((c + 1/2) * (1/cps)) in fp32 is
  // exact here (c < kMaxK * 64 = 1024 and cps <= 1024, so (c + 1/2) / cps is
  // at least 1/2048 from an integer, far beyond the product's rounding), and
  // takes three instructions where an integer division takes about twenty,
  // ahead of every row load
  static_assert(kMaxK * 64 <= 1024, "exact fp32 segment index");
  auto seg_div = [&](int c) { return (int)(((float)c + 0.5f) * a.seg_inv); };
  auto locate = [&](int c, int& sg, int& e0) {
    sg = cps > 0 ? min(seg_div(c), nseg - 1) : seg_of(st, nseg, c);
    e0 = (c - (cps > 0 ? sg * cps : st.start[sg])) * EPC;
  };
  auto klo = [&](int sg) { return AFF ? sg * a.seg_len : st.klo[sg]; };
  auto x_at = [&](int sg, int e0) -> const char* {
    return AFF ? a.x + xrow + sg * a.xs + (int64_t)e0 * ES : a.x + st.xoff[sg] + (int64_t)e0 * ES;
  };
  auto y_at = [&](int sg, int e0) -> char* {
    return AFF ? a.y + yrow + sg * a.ys + (int64_t)e0 * esy
               : a.y + st.yoff[sg] + ((int64_t)ri.row * st.len[sg] + e0) * esy;
  };
  auto w_at = [&](int sg) -> const char* { return AFF ? a.w + a.wbase + sg * a.ws : a.w + st.woff[sg]; };

  uint4 v[K];
  int seg[K], e0s[K];
  bool vis[K];
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const int c = cbase + k * 64 + lane;
    vis[k] = false;
    seg[k] = 0;
    e0s[k] = 0;
    v[k] = make_uint4(0, 0, 0, 0);
    if (c < total) {
      int sg, e0;  // e0: element index inside the segment
      locate(c, sg, e0);
      seg[k] = sg;
      e0s[k] = e0;
      vis[k] = active && (!(SOFTMAX && a.causal) || klo(sg) + e0 <= qpos);
      if (vis[k]) v[k] = *reinterpret_cast<const uint4*>(x_at(sg, e0));
    }
  }
  // Causal softmax: chunks wholly after the row's query position are zeros
  // of the output whatever the row's max and sum, so they are stored now,
  // while the row's loads are in flight, rather than after the reduction
  if constexpr (SOFTMAX) {
    if (a.causal && active) {
      auto store_zeros = [&](auto stream_tag) {
        constexpr bool STREAM = decltype(stream_tag)::value;
#pragma unroll
        for (int k = 0; k < K; ++k) {
          const int c = cbase + k * 64 + lane;
          if (c >= total || vis[k]) continue;
          char* yp = y_at(seg[k], e0s[k]);  // the chunk's EPC outputs, stored as write_row stores them
          if ((a.dt_y == EA_BF16 && ES == 2) || (a.dt_y == EA_F32 && ES == 4)) {
            store_out<STREAM>(yp, make_uint4(0, 0, 0, 0));
          } else {
#pragma unroll
            for (int i = 0; i < EPC; ++i) st_elem(yp, i, a.dt_y, 0.0f);
          }
        }
      };
      if (a.stream_out) store_zeros(std::true_type{});
      else store_zeros(std::false_type{});
    }
  }
  // RMSNorm weights.  On the affine layout with bf16 weights each lane loads
  // the weights of its own chunks into registers next to the row's loads
  // (L2 hits after the first rows); otherwise every wave of the workgroup
  // helps stage them in LDS while the row's loads are in flight.
  constexpr bool WREG = !SOFTMAX && AFF && ES == 2;
  uint4 wv[WREG ? K : 1];
  if constexpr (WREG) {
    if (a.dt_w == EA_BF16) {
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const int c = cbase + k * 64 + lane;
        wv[k] = make_uint4(0, 0, 0, 0);
        if (c < total && active) wv[k] = *reinterpret_cast<const uint4*>(w_at(seg[k]) + (int64_t)e0s[k] * 2);
      }
    }
  }
  if (!SOFTMAX && !(WREG && a.dt_w == EA_BF16)) {
    for (int c = threadIdx.x; c < total; c += kThreads) {
      int sg, e0;
      if constexpr (AFF) {
        sg = seg_div(c);
        e0 = (c - sg * cps) * EPC;
      } else {
        // the segment table of the wave that owns this chunk's row does not
        // matter: the weights depend only on the group, shared by the task
        locate(c, sg, e0);
      }
      const char* wb = w_at(sg);
      if (a.dt_w == EA_BF16 && EPC == 8) {  // one 16-byte load: 8 bf16 weights
        float f[8];
        unpack<uint16_t>(*reinterpret_cast<const uint4*>(wb + (int64_t)e0 * 2), f);
        *reinterpret_cast<float4*>(sw + c * EPC) = make_float4(f[0], f[1], f[2], f[3]);
        *reinterpret_cast<float4*>(sw + c * EPC + 4) = make_float4(f[4], f[5], f[6], f[7]);
      } else {
#pragma unroll
        for (int i = 0; i < EPC; ++i) sw[c * EPC + i] = ld_elem(wb, e0 + i, a.dt_w);
      }
    }
    __syncthreads();
  }
  if (WPR == 1 && !active) return;  // (split rows: every wave meets the barrier below)
  float scale = 0.0f, m = 0.0f;
  // softmax rows of at most 4 chunks per lane keep their exponentials from
  // the sum for the output, instead of computing them a second time
  constexpr bool KEEP = SOFTMAX && K <= 4;
  float ex[KEEP ? K : 1][KEEP ? 8 : 1];
#pragma unroll
  for (int k = 0; k < (KEEP ? K : 1); ++k)
#pragma unroll
    for (int i = 0; i < (KEEP ? 8 : 1); ++i) ex[k][i] = 0.0f;
  if constexpr (KEEP) {
    // Scores to the log2 domain once, kept in registers; the causal mask
    // (-inf, whose exponential is an exact 0) only where a lane's chunk
    // reaches past the row's query position, at most one chunk per row; the
    // max; then 2^(s - m) with one FMA and one exp per element.
    constexpr float kLog2e = 1.4426950408889634f;
    float part = -INFINITY;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      if (!vis[k]) continue;
      float f[8];
      unpack<XT>(v[k], f);
#pragma unroll
      for (int i = 0; i < EPC; ++i) ex[k][i] = f[i];
      if (a.causal) {
        const int k0 = klo(seg[k]) + e0s[k];
        if (__any(k0 + EPC - 1 > qpos)) {
#pragma unroll
          for (int i = 0; i < EPC; ++i) ex[k][i] = k0 + i <= qpos ? ex[k][i] : -INFINITY;
        }
      }
#pragma unroll
      for (int i = 0; i < EPC; ++i) part = fmaxf(part, ex[k][i]);
    }
    m = wave_max(part);
    const float mb = m == -INFINITY ? 0.0f : m * kLog2e;  // all entries -inf: every term 0
    float l = 0.0f;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      if (!vis[k]) continue;
#pragma unroll
      for (int i = 0; i < EPC; ++i) {
        ex[k][i] = __builtin_amdgcn_exp2f(fmaf(ex[k][i], kLog2e, -mb));
        l += ex[k][i];
      }
    }
    l = wave_sum(l);
    scale = m == -INFINITY ? 0.0f : 1.0f / l;
  } else {
  // local partials, then the aggregation across lanes
  float part = SOFTMAX ? -INFINITY : 0.0f;
  if constexpr (!SOFTMAX && ES == 2) {
    // bf16 sum of squares straight from the packed pairs: one v_dot2c_f32_bf16
    // per two elements (the bf16 products are exact in fp32), in four
    // running sums, one per 4-byte word of the chunk
    float p4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int k = 0; k < K; ++k) {
      if (!vis[k]) continue;
      const uint32_t w[4] = {v[k].x, v[k].y, v[k].z, v[k].w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bf16x2_t h = __builtin_bit_cast(bf16x2_t, w[i]);
        p4[i] = __builtin_amdgcn_fdot2_f32_bf16(h, h, p4[i], false);
      }
    }
    part = (p4[0] + p4[1]) + (p4[2] + p4[3]);
  } else {
#pragma unroll
  for (int k = 0; k < K; ++k) {
    if (!vis[k]) continue;
    float f[8];
    unpack<XT>(v[k], f);
    const int k0 = klo(seg[k]) + e0s[k];
#pragma unroll
    for (int i = 0; i < EPC; ++i) {
      if constexpr (SOFTMAX) {
        const bool ok = !a.causal || k0 + i <= qpos;
        part = ok ? fmaxf(part, f[i]) : part;
      } else {
        part += f[i] * f[i];
      }
    }
  }
  }
  if constexpr (SOFTMAX) {
    m = wave_max(part);
    float l = 0.0f;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      if (!vis[k]) continue;
      float f[8];
      unpack<XT>(v[k], f);
      const int k0 = klo(seg[k]) + e0s[k];
#pragma unroll
      for (int i = 0; i < EPC; ++i) {
        const bool ok = !a.causal || k0 + i <= qpos;
        l += ok ? __expf(f[i] - m) : 0.0f;
      }
    }
    l = wave_sum(l);
    scale = m == -INFINITY ? 0.0f : 1.0f / l;
  } else {
    float ss = wave_sum(part);
    if constexpr (WPR == 2) {  // the row's two halves, first half first
      if (lane == 0) s_half[wid] = ss;
      __syncthreads();
      ss = s_half[2 * wrow] + s_half[2 * wrow + 1];
    }
    scale = 1.0f / sqrtf(ss / (float)a.row_len + a.eps);
  }
  }
  if (WPR == 2 && !active) return;  // after the barrier: a wave past the task's rows writes nothing
  // write the row, under the output store policy (one branch around the
  // whole loop, see store_out)
  auto write_row = [&](auto stream_tag) {
    constexpr bool STREAM = decltype(stream_tag)::value;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int c = cbase + k * 64 + lane;
      if (c >= total) continue;
      if (SOFTMAX && a.causal && !vis[k]) continue;  // stored as zeros above
      const int sg = seg[k];
      const int e0 = e0s[k];
      float f[8];
      if constexpr (!KEEP) unpack<XT>(v[k], f);
      float o[8];
      if constexpr (KEEP) {  // masked and invisible entries hold exact zeros
#pragma unroll
        for (int i = 0; i < EPC; ++i) o[i] = vis[k] ? ex[k][i] * scale : 0.0f;
      } else if constexpr (SOFTMAX) {
        const int k0 = klo(sg) + e0;
#pragma unroll
        for (int i = 0; i < EPC; ++i) {
          const bool ok = vis[k] && (!a.causal || k0 + i <= qpos);
          o[i] = ok ? __expf(f[i] - m) * scale : 0.0f;
        }
      } else if (WREG && a.dt_w == EA_BF16) {
        float wf[8];
        unpack<uint16_t>(wv[WREG ? k : 0], wf);
#pragma unroll
        for (int i = 0; i < EPC; ++i) o[i] = wf[i] * (f[i] * scale);
      } else {
#pragma unroll
        for (int i = 0; i < EPC; ++i) o[i] = sw[c * EPC + i] * (f[i] * scale);
      }
      char* yp = y_at(sg, e0);
      if (a.dt_y == EA_BF16 && ES == 2) {
        uint4 pk;
        uint32_t* w = reinterpret_cast<uint32_t*>(&pk);
#pragma unroll
        for (int i = 0; i < 4; ++i) w[i] = pack_bf16x2(o[2 * i], o[2 * i + 1]);
        store_out<STREAM>(yp, pk);
      } else if (a.dt_y == EA_F32 && ES == 4) {
        store_out<STREAM>(yp, make_uint4(__float_as_uint(o[0]), __float_as_uint(o[1]), __float_as_uint(o[2]),
                                         __float_as_uint(o[3])));
      } else {
#pragma unroll
        for (int i = 0; i < EPC; ++i) st_elem(yp, i, a.dt_y, o[i]);
      }
    }
  };
  if (a.stream_out) write_row(std::true_type{});
  else write_row(std::false_type{});
}

// ---------------------------------------------------------------------------
// scalar path: any segment lengths, any row length; re-reads the row
// ---------------------------------------------------------------------------
template <bool SOFTMAX>
__global__ __launch_bounds__(kThreads) void rows_scalar_kernel(RowArgs a) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  if (wid >= a.tasks[blockIdx.x].nrows) return;
  const RowInfo ri = row_info(a, wid);
  const int d_last = a.rank - 1;
  auto visit = [&](auto&& fn) {
    for (int s = 0; s < ri.nseg; ++s) {
      const int32_t* tp = a.tuples + (int64_t)(ri.t0 + s) * a.tuple_stride;
      const DevBlk& xb = a.blk_x[tp[1]];
      const int L = xb.ext[d_last];
      const char* xbase = a.x + xb.off;
      for (int e = lane; e < L; e += 64) {
        const int64_t idx = (int64_t)ri.row * L + e;
        const bool ok = !(SOFTMAX && a.causal) || xb.lo[d_last] + e <= ri.qpos;
        fn(tp, idx, e, ok, ok ? ld_elem(xbase, idx, a.dt_x) : 0.0f);
      }
    }
  };
  if constexpr (SOFTMAX) {
    float m = -INFINITY;
    visit([&](const int32_t*, int64_t, int, bool ok, float x) { m = ok ? fmaxf(m, x) : m; });
    m = wave_max(m);
    float l = 0.0f;
    visit([&](const int32_t*, int64_t, int, bool ok, float x) { l += ok ? __expf(x - m) : 0.0f; });
    l = wave_sum(l);
    const float inv = m == -INFINITY ? 0.0f : 1.0f / l;
    visit([&](const int32_t* tp, int64_t idx, int, bool ok, float x) {
      st_elem(a.y + a.blk_y[tp[0]].off, idx, a.dt_y, ok ? __expf(x - m) * inv : 0.0f);
    });
  } else {
    float ss = 0.0f;
    visit([&](const int32_t*, int64_t, int, bool, float x) { ss += x * x; });
    ss = wave_sum(ss);
    const float inv = 1.0f / sqrtf(ss / (float)a.row_len + a.eps);
    visit([&](const int32_t* tp, int64_t idx, int e, bool, float x) {
      const float w = ld_elem(a.w + a.blk_w[tp[2]].off, e, a.dt_w);
      st_elem(a.y + a.blk_y[tp[0]].off, idx, a.dt_y, w * (x * inv));
    });
  }
}

template <typename XT, bool SOFTMAX, int K>
void launch_vec(const RowArgs& a, dim3 grid, dim3 block, hipStream_t s) {
  if (a.affine) hipLaunchKernelGGL((rows_vec_kernel<XT, SOFTMAX, K, true>), grid, block, 0, s, a);
  else hipLaunchKernelGGL((rows_vec_kernel<XT, SOFTMAX, K, false>), grid, block, 0, s, a);
}

// bf16 RMSNorm rows of 8K+ bf16 chunks on the affine layout with bf16
// weights: two wavefronts per row (kMaxK / 2 chunks per lane each)
bool split_rows(const RowArgs& a, int64_t chunks, bool softmax) {
  return !softmax && a.affine && a.dt_x == EA_BF16 && a.dt_w == EA_BF16 && chunks > (kMaxK / 2) * 64;
}

template <typename XT, bool SOFTMAX>
void launch_vec_k(const RowArgs& a, int64_t chunks, dim3 grid, dim3 block, hipStream_t s) {
  if constexpr (!SOFTMAX && sizeof(XT) == 2) {
    if (split_rows(a, chunks, SOFTMAX)) {
      hipLaunchKernelGGL((rows_vec_kernel<XT, false, kMaxK / 2, true, 2>), grid, dim3(block.x * 2), 0, s, a);
      return;
    }
  }
  if (chunks <= 4 * 64) launch_vec<XT, SOFTMAX, 4>(a, grid, block, s);
  else if (chunks <= 8 * 64) launch_vec<XT, SOFTMAX, 8>(a, grid, block, s);
  else launch_vec<XT, SOFTMAX, kMaxK>(a, grid, block, s);
}

template <bool SOFTMAX>
hipError_t launch_rows(const RowArgs& a, hipStream_t s) {
  if (a.n_rowtasks == 0) return hipSuccess;
  const dim3 grid((uint32_t)a.n_rowtasks), block(kThreads);
  if (a.vec) {
    const int64_t chunks = (int64_t)a.row_len * (a.dt_x == EA_BF16 ? 2 : 4) / 16;
    if (a.dt_x == EA_BF16) launch_vec_k<uint16_t, SOFTMAX>(a, chunks, grid, block, s);
    else launch_vec_k<float, SOFTMAX>(a, chunks, grid, block, s);
  } else {
    hipLaunchKernelGGL((rows_scalar_kernel<SOFTMAX>), grid, block, 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_rmsnorm(const RowArgs& a, hipStream_t s) { return launch_rows<false>(a, s); }
hipError_t launch_softmax(const RowArgs& a, hipStream_t s) { return launch_rows<true>(a, s); }

// Whether a row layout fits the register path: every segment a multiple of
// 16 bytes, at most kMaxSeg segments and kMaxK chunks per lane.
bool rows_vec_ok(int64_t row_len, int64_t max_segments, bool seg_aligned, int es) {
  return seg_aligned && max_segments <= kMaxSeg && row_len * es <= (int64_t)kMaxK * 64 * 16;
}

}  // namespace ea
