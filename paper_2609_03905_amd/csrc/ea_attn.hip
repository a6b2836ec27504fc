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
// workgroup is 4 waves x 32 query rows.  Per 128-key chunk:
//   * K [key][d] (bf16) and V^T [d][key] (converted to fp16 while staging,
//     transposed in registers, 4-key units XOR-swizzled against bank
//     conflicts) are staged in LDS;
//   * S^T = K Q^T on bf16 MFMA 32x32x16 (Q^T from registers), so each lane
//     holds the scores of one query: the row max and sum need one exchange
//     between lanes l and l^32;
//   * P = 2^(S - m) is split into fp16 P_hi + P_lo (about 22 significant
//     bits) and O^T += V^T P_hi^T + V^T P_lo^T runs on fp16 MFMA, with the
//     MFMA's k order matched to the accumulator layout of S^T.
// A group whose tuples are split across units writes partial (m, l, O) to the
// plan's scratch; the last unit to arrive (device-scope counter, no waiting)
// merges the partials in tuple order and stores the output block rows.
#include "ea_device.h"

namespace ea {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int D = 128;   // head dim
constexpr int KC = 128;  // keys per staged chunk
constexpr int KP = 136;  // K row pitch in LDS (halves)
constexpr int VP = 136;  // V^T row pitch in LDS (halves)
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ f32x16_t mfma_bf16(const uint4& a, const uint4& b, const f32x16_t& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                  c, 0, 0, 0);
}

__device__ __forceinline__ f32x16_t mfma_f16(const uint4& a, const uint4& b, const f32x16_t& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b), c,
                                                 0, 0, 0);
}

__device__ __forceinline__ uint32_t pack_f16x2(float a, float b) {
  return (uint32_t)f32_to_f16(a) | ((uint32_t)f32_to_f16(b) << 16);
}

// bf16 pair (one 32-bit word) -> two fp16 values, as floats first.
__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ uint32_t word(const uint4& v, int w) {
  return w == 0 ? v.x : w == 1 ? v.y : w == 2 ? v.z : v.w;
}

__global__ __launch_bounds__(kThreads, 1) void attn_kernel(const AttnArgs p) {
  __shared__ __attribute__((aligned(16))) uint16_t sK[KC * KP];
  __shared__ __attribute__((aligned(16))) uint16_t sV[D * VP];
  __shared__ int s_last;

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int g = lane >> 5, lq = lane & 31;
  const AttnUnit u = p.units[blockIdx.x];
  const int32_t* __restrict__ tuples = p.tuples;
  const int32_t gb = p.goff[u.group], ge = p.goff[u.group + 1];
  const int n = ge - gb;
  const int tb = gb + (int)(((int64_t)u.part * n) / u.n_parts);
  const int te = gb + (int)(((int64_t)(u.part + 1) * n) / u.n_parts);
  const int qd = p.q_dim, kd = p.k_dim;

  // every tuple of the group carries the same output and Q blocks
  const DevBlk& qblk = p.blk_q[tuples[(int64_t)gb * 4 + 1]];
  const DevBlk& oblk = p.blk_o[tuples[(int64_t)gb * 4 + 0]];
  const int q_lo = qblk.lo[qd];
  const int row = u.q0 + wid * 32 + lq;        // this lane's query row inside the block
  const int qpos = q_lo + row;                 // its position
  const int qpos_wave_max = q_lo + u.q0 + wid * 32 + 31;
  const int qpos_tile_max = q_lo + u.q0 + 127;
  const float sc = p.scale * kLog2e;
  const bool causal = p.causal != 0;

  // Q^T operand: lane holds Q[row][16 s + 8 g .. + 7] for s = 0..7
  uint4 qreg[8];
  {
    const char* qrow = p.q + qblk.off + (int64_t)row * D * 2;
#pragma unroll
    for (int s = 0; s < 8; ++s) qreg[s] = *reinterpret_cast<const uint4*>(qrow + (16 * s + 8 * g) * 2);
  }

  f32x16_t acc_o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc_o[i] = f32x16_t{};
  float m = -INFINITY, l = 0.0f;

  for (int t = tb; t < te; ++t) {
    const int32_t* tp = tuples + (int64_t)t * 4;
    const DevBlk& kb = p.blk_k[tp[2]];
    const DevBlk& vb = p.blk_v[tp[3]];
    const int k_lo = kb.lo[kd], k_ext = kb.ext[kd];
    const char* kbase = p.k + kb.off;
    const char* vbase = p.v + vb.off;
    for (int c0 = 0; c0 < k_ext; c0 += KC) {
      const int key0 = k_lo + c0;
      if (causal && key0 > qpos_tile_max) break;  // this and later chunks are masked for the whole tile
      __syncthreads();  // previous chunk's LDS reads are done
      // ---- stage K chunk: rows c0..c0+127, 16-byte pieces
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int c = tid + kThreads * i;
        const int r = c >> 4, cc = c & 15;
        *reinterpret_cast<uint4*>(sK + r * KP + cc * 8) =
            *reinterpret_cast<const uint4*>(kbase + ((int64_t)(c0 + r) * D + cc * 8) * 2);
        if (i == 3) __builtin_amdgcn_sched_barrier(0);  // at most 4 pieces in flight per thread
      }
      // ---- stage V^T chunk in fp16: thread takes 4 keys x 8 dims, twice
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int blk = tid + kThreads * i;
        const int dg = blk & 15, kg = blk >> 4;
        uint4 v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r)
          v[r] = *reinterpret_cast<const uint4*>(vbase + ((int64_t)(c0 + 4 * kg + r) * D + 8 * dg) * 2);
        const int phys = kg ^ dg;  // swizzled 4-key unit
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int w = j >> 1;
          float f[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) f[r] = (j & 1) ? hi_bf16(word(v[r], w)) : lo_bf16(word(v[r], w));
          uint2 o;
          o.x = pack_f16x2(f[0], f[1]);
          o.y = pack_f16x2(f[2], f[3]);
          *reinterpret_cast<uint2*>(sV + (8 * dg + j) * VP + 4 * phys) = o;
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      __syncthreads();
      if (causal && key0 > qpos_wave_max) continue;  // the whole wave is masked in this chunk

      // ---- S^T = K Q^T for 128 keys x this wave's 32 queries
      f32x16_t acc_s[4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) acc_s[kt] = f32x16_t{};
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        uint4 a[4];
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
          a[kt] = *reinterpret_cast<const uint4*>(sK + (32 * kt + lq) * KP + 16 * s + 8 * g);
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) acc_s[kt] = mfma_bf16(a[kt], qreg[s], acc_s[kt]);
        __builtin_amdgcn_sched_barrier(0);  // keep operand reads from piling up across steps
      }
      // ---- scale, mask, online softmax (log2 domain)
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float sv = acc_s[kt][r] * sc;
          if (causal) {
            const int kpos = key0 + 32 * kt + 8 * (r >> 2) + 4 * g + (r & 3);
            sv = kpos > qpos ? -INFINITY : sv;
          }
          acc_s[kt][r] = sv;
          mx = fmaxf(mx, sv);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m, mx);
      const float m_use = m_new == -INFINITY ? 0.0f : m_new;
      const float alpha = exp2f(m - m_use);
      float rs = 0.0f;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float pv = exp2f(acc_s[kt][r] - m_use);
          acc_s[kt][r] = pv;
          rs += pv;
        }
      rs += __shfl_xor(rs, 32, 64);
      l = l * alpha + rs;
      m = m_new;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc_o[dt][r] *= alpha;

      // ---- O^T += V^T P^T (fp16).  MFMA k index 8 g + j maps to key
      // 32 kt + 16 h + 4 g + j (j < 4) or 32 kt + 16 h + 8 + 4 g + (j - 4).
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          // P = P_hi + P_lo, both fp16 (about 22 significant bits together)
          uint32_t hi[4], lo[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float p0 = acc_s[kt][8 * h + 2 * e], p1 = acc_s[kt][8 * h + 2 * e + 1];
            const uint16_t h0 = f32_to_f16(p0), h1 = f32_to_f16(p1);
            hi[e] = (uint32_t)h0 | ((uint32_t)h1 << 16);
            lo[e] = pack_f16x2(p0 - f16_to_f32(h0), p1 - f16_to_f32(h1));
          }
          const uint4 pb = make_uint4(hi[0], hi[1], hi[2], hi[3]);
          const uint4 pl = make_uint4(lo[0], lo[1], lo[2], lo[3]);
          const int u0 = 8 * kt + 4 * h + g, u1 = u0 + 2;
#pragma unroll
          for (int dt = 0; dt < 4; ++dt) {
            const int d = 32 * dt + lq;
            const int sw = (d >> 3) & 15;
            const uint2 a0 = *reinterpret_cast<const uint2*>(sV + d * VP + 4 * (u0 ^ sw));
            const uint2 a1 = *reinterpret_cast<const uint2*>(sV + d * VP + 4 * (u1 ^ sw));
            const uint4 va = make_uint4(a0.x, a0.y, a1.x, a1.y);
            acc_o[dt] = mfma_f16(va, pb, acc_o[dt]);
            acc_o[dt] = mfma_f16(va, pl, acc_o[dt]);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
    }
  }

  // ---- epilogue.  acc_o[dt] register r of lane (lq, g) holds O^T row
  // d = 32 dt + 8 (r/4) + 4 g + r%4, column = this lane's query.
  if (u.slot < 0) {
    const float inv = l > 0.0f ? 1.0f / l : 0.0f;
    char* orow = p.o + oblk.off;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int d = 32 * dt + 8 * rr + 4 * g;
        const int64_t idx = (int64_t)row * D + d;
        const float o0 = acc_o[dt][4 * rr] * inv, o1 = acc_o[dt][4 * rr + 1] * inv;
        const float o2 = acc_o[dt][4 * rr + 2] * inv, o3 = acc_o[dt][4 * rr + 3] * inv;
        if (p.dt_o == EA_BF16) {
          uint2 w;
          w.x = (uint32_t)f32_to_bf16(o0) | ((uint32_t)f32_to_bf16(o1) << 16);
          w.y = (uint32_t)f32_to_bf16(o2) | ((uint32_t)f32_to_bf16(o3) << 16);
          *reinterpret_cast<uint2*>(orow + idx * 2) = w;
        } else {
          *reinterpret_cast<float4*>(orow + idx * 4) = make_float4(o0, o1, o2, o3);
        }
      }
    return;
  }

  // ---- split group: write this unit's partial, the last unit merges
  {
    float* po = p.part_o + (int64_t)u.slot * 128 * D;
    const int rt = wid * 32 + lq;  // row inside the tile
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int d = 32 * dt + 8 * rr + 4 * g;
        store_agent2(po + rt * D + d, acc_o[dt][4 * rr], acc_o[dt][4 * rr + 1]);
        store_agent2(po + rt * D + d + 2, acc_o[dt][4 * rr + 2], acc_o[dt][4 * rr + 3]);
      }
    if (g == 0) store_agent2(p.part_ml + ((int64_t)u.slot * 128 + rt) * 2, m, l);
  }
  drain_vmem();
  __syncthreads();
  if (tid == 0) s_last = arrive_agent(p.counters + u.counter) == u.n_parts - 1;
  __syncthreads();
  if (!s_last) return;
  {
    const int rt = tid >> 1, dlo = (tid & 1) * 64;
    float M = -INFINITY;
    for (int q = 0; q < u.n_parts; ++q) M = fmaxf(M, load_agent(p.part_ml + ((int64_t)(u.first_slot + q) * 128 + rt) * 2));
    const float Mu = M == -INFINITY ? 0.0f : M;
    float L = 0.0f;
    for (int q = 0; q < u.n_parts; ++q) {
      const float2 ml = load_agent2(p.part_ml + ((int64_t)(u.first_slot + q) * 128 + rt) * 2);
      L += ml.y * exp2f(ml.x - Mu);
    }
    const float inv = L > 0.0f ? 1.0f / L : 0.0f;
    const int64_t orow_idx = (int64_t)(u.q0 + rt) * D;
    char* obase = p.o + oblk.off;
    for (int d = dlo; d < dlo + 64; d += 4) {
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int q = 0; q < u.n_parts; ++q) {
        const int64_t sl = u.first_slot + q;
        const float w = exp2f(load_agent(p.part_ml + (sl * 128 + rt) * 2) - Mu);
        const float2 v0 = load_agent2(p.part_o + (sl * 128 + rt) * D + d);
        const float2 v1 = load_agent2(p.part_o + (sl * 128 + rt) * D + d + 2);
        acc.x += v0.x * w;
        acc.y += v0.y * w;
        acc.z += v1.x * w;
        acc.w += v1.y * w;
      }
      const float o0 = acc.x * inv, o1 = acc.y * inv, o2 = acc.z * inv, o3 = acc.w * inv;
      if (p.dt_o == EA_BF16) {
        uint2 w;
        w.x = (uint32_t)f32_to_bf16(o0) | ((uint32_t)f32_to_bf16(o1) << 16);
        w.y = (uint32_t)f32_to_bf16(o2) | ((uint32_t)f32_to_bf16(o3) << 16);
        *reinterpret_cast<uint2*>(obase + (orow_idx + d) * 2) = w;
      } else {
        *reinterpret_cast<float4*>(obase + (orow_idx + d) * 4) = make_float4(o0, o1, o2, o3);
      }
    }
  }
  if (tid == 0) reset_agent(p.counters + u.counter);  // ready for the next call (stream-ordered)
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.n_units == 0) return hipSuccess;
  hipLaunchKernelGGL(attn_kernel, dim3((uint32_t)a.n_units), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace ea
