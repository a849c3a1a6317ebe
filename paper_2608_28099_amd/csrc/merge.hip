// Merge of the split-attention partials with the soft keys themselves
// (Sec. 3.3, Eq. 1-3).  Per query row the merge computes the soft keys visible
// to it (causal: key j' <= j) in fp32 and combines them with the splits' partials
// (running max m_s in log2 units, sum l_s, unnormalised O_s) by the
// log-sum-exp rule
//   M = max(m_soft, max_s m_s),  L = l_soft 2^(m_soft-M) + sum_s l_s 2^(m_s-M),
//   O = (O_soft 2^(m_soft-M) + sum_s O_s 2^(m_s-M)) / L.
#include "common.h"
#include "kernels.h"

namespace sp {
namespace {

// N consecutive soft operands as stored by rope_scatter (fp32, or bf16 hi + lo
// parts summed in fp32), N a multiple of 8, with 16-byte loads.
template <typename TI, int N>
__device__ __forceinline__ void soft_load_vec(const void* hi, const void* lo, int64_t idx, float (&v)[N]) {
  if constexpr (sizeof(TI) == 4) {
#pragma unroll
    for (int i = 0; i < N; i += 4) {
      const float4 x = *reinterpret_cast<const float4*>((const float*)hi + idx + i);
      v[i] = x.x; v[i + 1] = x.y; v[i + 2] = x.z; v[i + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < N; i += 8) {
      const bf16x8 h = *reinterpret_cast<const bf16x8*>((const bf16*)hi + idx + i);
      const bf16x8 l = *reinterpret_cast<const bf16x8*>((const bf16*)lo + idx + i);
#pragma unroll
      for (int t = 0; t < 8; ++t) v[i + t] = (float)h[t] + (float)l[t];
    }
  }
}

// One workgroup per (sequence b, KV head g, block of rw consecutive soft rows
// with queries of one task): its rows see soft keys [j_lo, j] of their task (at
// most 64), and the workgroup stages the union, [j_lo, j of its last row], once
// in LDS as fp32 (keys and values; from the stored operands: fp32, or bf16
// hi + lo), with 16-byte loads.  Its rw G query rows are dealt to the waves; a
// wave's first row's split partials and query are requested before the
// staging, so the two round trips overlap.  Soft scores are fp32, 16 keys per pass: lane l takes
// key j_lo + 16 ci + (l & 15) over head dims [(l >> 4) hd/4, +hd/4), and two
// shuffles add the four dim groups.  Then P V (lane l owns output dims
// l DPL .. l DPL + DPL - 1, DPL = hd / 64, each key's probability broadcast
// from its lane), and the splits folded in with a running maximum
// (log-sum-exp rule), four at a time.  TO: output type; TI: soft operand storage.
template <typename TO, typename TI, int DPL>
__global__ __launch_bounds__(256) void merge_splits(const MergeParams p) {
  constexpr int C = 4;                       // splits per batch of loads
  constexpr int HD = 64 * DPL, DG = HD / 4;  // head dim; dims per lane group in the scores
  extern __shared__ float kvs[];             // [nk][HD] keys, then [nk][HD] values
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, nw = blockDim.x >> 6;
  const int g = blockIdx.y, b = blockIdx.z;
  if (p.err && *p.err) return;
  const int n = clamp_len(p.seq_lens, b, p.max_seq_len);
  const int ns = n > 0 ? (n + p.split_len - 1) / p.split_len : 1;
  const int bpt = (p.q_per_task + p.rw - 1) / p.rw;                // row blocks per task
  const int task = blockIdx.x / bpt, q0 = (blockIdx.x % bpt) * p.rw;
  const int nq = min(p.rw, p.q_per_task - q0);                     // soft rows of this workgroup
  const int nrows = nq * p.group;                                  // its query rows
  const int j_lo = task * p.k_task;                                // the task's first soft key
  const int nk_all = p.q_first + q0 + nq + p.step;                 // keys [j_lo, j of the last row]
  const int i0 = lane * DPL, kl = lane & 15, grp = lane >> 4;

  // inputs of one query row: split partials (a batch of C) and the query
  struct RowIn {
    float2 ml[C];
    float ov[C][DPL];
    float qg[DG];
  };
  auto row_qi = [&](int r) __attribute__((always_inline)) { return task * p.q_per_task + q0 + r / p.group; };
  auto row_base = [&](int r) __attribute__((always_inline)) {
    return ((int64_t)b * p.n_kv + g) * p.max_splits * p.r_alloc + row_qi(r) * p.group + r % p.group;
  };
  auto load_splits = [&](int64_t base, int s0, RowIn& in) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < C; ++c) {
      const int64_t row = base + (int64_t)min(s0 + c, ns - 1) * p.r_alloc;
      in.ml[c] = p.ml_part[row];
#pragma unroll
      for (int d = 0; d < DPL; ++d) in.ov[c][d] = p.o_part[row * HD + i0 + d];
    }
  };
  auto load_row = [&](int r, RowIn& in) __attribute__((always_inline)) {
    load_splits(row_base(r), 0, in);
    const int64_t qo = (((int64_t)b * p.n_kv + g) * p.r_alloc + row_qi(r) * p.group + r % p.group) * HD;
    soft_load_vec<TI, DG>(p.q, p.q_lo, qo + grp * DG, in.qg);
  };
  RowIn cur;
  if (wave < nrows) load_row(wave, cur);
  bool oor = false;

  // stage the keys and values of the workgroup's window
  const int64_t ko = (((int64_t)b * p.n_kv + g) * p.ks + j_lo) * HD;                      // [ks][hd]
  const int64_t vo = (((p.per_seq ? (int64_t)b * p.n_kv : 0) + g) * p.ks + j_lo) * HD;  // [ks][hd]
  float* ks_ = kvs;
  float* vs_ = kvs + nk_all * HD;
  for (int e = threadIdx.x * 8; e < nk_all * HD; e += blockDim.x * 8) {
    float kx[8], vx[8];
    soft_load_vec<TI, 8>(p.k_soft, p.k_soft_lo, ko + e, kx);
    soft_load_vec<TI, 8>(p.v_soft, p.v_soft_lo, vo + e, vx);
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      ks_[e + t] = kx[t];
      vs_[e + t] = vx[t];
    }
  }
  __syncthreads();

  for (int r = wave; r < nrows; r += nw) {
    if (r != wave) load_row(r, cur);
    const int qi = row_qi(r), hq = r % p.group;
    const int nk = p.q_first + qi % p.q_per_task + p.step + 1;  // keys [j_lo, j] of this row
    const int nch = (nk + 15) >> 4;
    float sc[4];
#pragma unroll
    for (int ci = 0; ci < 4; ++ci) {
      sc[ci] = -INFINITY;
      if (ci < nch) {
        const int t = 16 * ci + kl;  // key j_lo + t
        const float* kr = ks_ + min(t, nk - 1) * HD + grp * DG;
        float part = 0.f;
#pragma unroll
        for (int d = 0; d < DG; d += 4) {
          const float4 k4 = *reinterpret_cast<const float4*>(kr + d);
          part += cur.qg[d] * k4.x + cur.qg[d + 1] * k4.y + cur.qg[d + 2] * k4.z + cur.qg[d + 3] * k4.w;
        }
        part += __shfl_xor(part, 16);
        part += __shfl_xor(part, 32);
        if (t < nk) sc[ci] = part;
      }
    }
    float M = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));  // key j_lo is always visible: finite
    for (int o = 8; o > 0; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
    float pj[4], ls = 0.f;
#pragma unroll
    for (int ci = 0; ci < 4; ++ci) {
      pj[ci] = fast_exp2(sc[ci] - M);  // 0 for masked keys
      ls += pj[ci];
    }
    float L = ls;  // the 16 lanes of a group hold every key once
    for (int o = 8; o > 0; o >>= 1) L += __shfl_xor(L, o);
    float acc[DPL];
#pragma unroll
    for (int d = 0; d < DPL; ++d) acc[d] = 0.f;
#pragma unroll
    for (int ci = 0; ci < 4; ++ci) {
      if (ci < nch) {
        // all 16 slots, branch-free, so the LDS reads are in flight together
        // (slots past the window read its last key with weight 0)
#pragma unroll
        for (int c = 0; c < 16; ++c) {
          const float pk = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, pj[ci]), c));
          const float* vr = vs_ + min(16 * ci + c, nk - 1) * HD + i0;
#pragma unroll
          for (int d = 0; d < DPL; ++d) acc[d] += pk * vr[d];
        }
      }
    }
    // split partials, folded in with a running maximum
    const int64_t base = row_base(r);
    for (int s0 = 0; s0 < ns; s0 += C) {
      if (s0 > 0) load_splits(base, s0, cur);
      float mn = M;
#pragma unroll
      for (int c = 0; c < C; ++c)
        if (s0 + c < ns) mn = fmaxf(mn, cur.ml[c].x);
      const float alpha = fast_exp2(M - mn);
      L *= alpha;
#pragma unroll
      for (int d = 0; d < DPL; ++d) acc[d] *= alpha;
#pragma unroll
      for (int c = 0; c < C; ++c) {
        if (s0 + c < ns) {
          const float wgt = fast_exp2(cur.ml[c].x - mn);
          L += cur.ml[c].y * wgt;
#pragma unroll
          for (int d = 0; d < DPL; ++d) acc[d] += cur.ov[c][d] * wgt;
        }
      }
      M = mn;
    }
    const float inv = 1.0f / L;
    const int h = g * p.group + hq;
    TO* out = (TO*)p.out + ((int64_t)b * p.out_rows + p.out_off + qi) * ((int64_t)p.n_q * HD) +
              (int64_t)h * HD + i0;
#pragma unroll
    for (int d = 0; d < DPL; ++d) {
      out[d] = from_f32<TO>(acc[d] * inv);
      if constexpr (sizeof(TO) == 2) oor |= !(fabsf(acc[d] * inv) <= 65504.0f);
    }
  }
  // an fp16 output out of fp16's range (a convex combination of the values,
  // so only values out of range can cause it)
  if constexpr (sizeof(TO) == 2)
    if (__any(oor) && lane == 0 && p.status) atomicOr(p.status, kStatusRange);
}

}  // namespace

hipError_t launch_merge(DType dt, const MergeParams& p, int batch, hipStream_t s) {
  if (p.hd != 64 && p.hd != 128) return hipErrorInvalidValue;
  // widest key window: the last row with queries of a task sees q_first + q_per_task + step keys
  const int nk_max = p.q_first + p.q_per_task + p.step;
  if (nk_max > 64 || p.rows % p.group) return hipErrorInvalidValue;
  if (p.q_per_task < 1 || (p.rows / p.group) % p.q_per_task) return hipErrorInvalidValue;
  const int tasks = p.rows / p.group / p.q_per_task;
  // Soft rows per workgroup: the most (a power of two) that still leave
  // min_wgs workgroups (4 per compute unit).  Each workgroup stages its key
  // window once and then streams its rows' partials; measured against 1-16
  // workgroups per compute unit this was fastest on every workload (long
  // context: 32 us against 44 us at one soft row per workgroup; 27B shape:
  // 0.37 ms against 0.86 ms).
  MergeParams q = p;
  const int64_t min_wgs = p.min_wgs > 0 ? p.min_wgs : 1024;
  q.rw = 1;
  while (2 * q.rw <= p.q_per_task &&
         (int64_t)batch * p.n_kv * tasks * ((p.q_per_task + 2 * q.rw - 1) / (2 * q.rw)) >= min_wgs)
    q.rw *= 2;
  const int bpt = (p.q_per_task + q.rw - 1) / q.rw;
  const dim3 grid(tasks * bpt, p.n_kv, batch);
  const int rows_wg = q.rw * p.group;
  const dim3 block(64 * (rows_wg < 4 ? rows_wg : 4));
  const size_t lds = (size_t)2 * nk_max * p.hd * sizeof(float);  // its keys and values, fp32
  if (dt == kBF16) {  // the attention output feeds an fp16 MFMA
    if (p.hd == 128) hipLaunchKernelGGL((merge_splits<f16, bf16, 2>), grid, block, lds, s, q);
    else hipLaunchKernelGGL((merge_splits<f16, bf16, 1>), grid, block, lds, s, q);
  } else {
    if (p.hd == 128) hipLaunchKernelGGL((merge_splits<float, float, 2>), grid, block, lds, s, q);
    else hipLaunchKernelGGL((merge_splits<float, float, 1>), grid, block, lds, s, q);
  }
  return hipGetLastError();
}

}  // namespace sp
