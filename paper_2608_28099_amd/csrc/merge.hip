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

// One workgroup per (sequence b, KV head g, soft row with queries): its G
// query rows r = qi G + 0..G-1 see the same soft keys, [j_lo, j] of their task
// (at most 64), which the workgroup stages once in LDS as fp32 (keys and
// values; from the stored operands: fp32, or bf16 hi + lo), with 16-byte
// loads.  One wave per query row (looping when G exceeds the wave count).  A
// row's split partials and query are requested before the staging, so both
// round trips overlap.  Soft scores are fp32, 16 keys per pass: lane l takes
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
  const int qi = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  if (p.err && *p.err) return;
  const int n = clamp_len(p.seq_lens, b, p.max_seq_len);
  const int ns = n > 0 ? (n + p.split_len - 1) / p.split_len : 1;
  const int j_lo = (qi / p.q_per_task) * p.k_task;                 // the task's first soft key
  const int j = j_lo + p.q_first + qi % p.q_per_task + p.step;     // this soft row
  const int nk = j - j_lo + 1, nch = (nk + 15) >> 4;
  const int i0 = lane * DPL, kl = lane & 15, grp = lane >> 4;

  float2 ml[C];
  float ov[C][DPL];
  float qg[DG];
  auto load_splits = [&](int64_t base, int s0) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < C; ++c) {
      const int64_t row = base + (int64_t)min(s0 + c, ns - 1) * p.r_alloc;
      ml[c] = p.ml_part[row];
#pragma unroll
      for (int d = 0; d < DPL; ++d) ov[c][d] = p.o_part[row * HD + i0 + d];
    }
  };
  auto row_base = [&](int hq) __attribute__((always_inline)) {
    return ((int64_t)b * p.n_kv + g) * p.max_splits * p.r_alloc + qi * p.group + hq;
  };
  auto load_query = [&](int hq) __attribute__((always_inline)) {
    const int64_t qo = (((int64_t)b * p.n_kv + g) * p.r_alloc + qi * p.group + hq) * HD;
    soft_load_vec<TI, DG>(p.q, p.q_lo, qo + grp * DG, qg);
  };
  if (wave < p.group) {
    load_splits(row_base(wave), 0);
    load_query(wave);
  }

  // stage the window's keys and values
  const int64_t ko = (((int64_t)b * p.n_kv + g) * p.ks + j_lo) * HD;                      // [ks][hd]
  const int64_t vo = (((p.per_seq ? (int64_t)b * p.n_kv : 0) + g) * p.ks + j_lo) * HD;  // [ks][hd]
  float* ks_ = kvs;
  float* vs_ = kvs + nk * HD;
  for (int e = threadIdx.x * 8; e < nk * HD; e += blockDim.x * 8) {
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

  for (int hq = wave; hq < p.group; hq += nw) {
    const int64_t base = row_base(hq);
    if (hq != wave) {
      load_splits(base, 0);
      load_query(hq);
    }
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
          part += qg[d] * k4.x + qg[d + 1] * k4.y + qg[d + 2] * k4.z + qg[d + 3] * k4.w;
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
    for (int s0 = 0; s0 < ns; s0 += C) {
      if (s0 > 0) load_splits(base, s0);
      float mn = M;
#pragma unroll
      for (int c = 0; c < C; ++c)
        if (s0 + c < ns) mn = fmaxf(mn, ml[c].x);
      const float alpha = fast_exp2(M - mn);
      L *= alpha;
#pragma unroll
      for (int d = 0; d < DPL; ++d) acc[d] *= alpha;
#pragma unroll
      for (int c = 0; c < C; ++c) {
        if (s0 + c < ns) {
          const float wgt = fast_exp2(ml[c].x - mn);
          L += ml[c].y * wgt;
#pragma unroll
          for (int d = 0; d < DPL; ++d) acc[d] += ov[c][d] * wgt;
        }
      }
      M = mn;
    }
    const float inv = 1.0f / L;
    const int h = g * p.group + hq;
    TO* out = (TO*)p.out + ((int64_t)b * p.out_rows + p.out_off + qi) * ((int64_t)p.n_q * HD) +
              (int64_t)h * HD + i0;
#pragma unroll
    for (int d = 0; d < DPL; ++d) out[d] = from_f32<TO>(acc[d] * inv);
  }
}

}  // namespace

hipError_t launch_merge(DType dt, const MergeParams& p, int batch, hipStream_t s) {
  if (p.hd != 64 && p.hd != 128) return hipErrorInvalidValue;
  // widest key window: the last row with queries of a task sees q_first + q_per_task + step keys
  const int nk_max = p.q_first + p.q_per_task + p.step;
  if (nk_max > 64 || p.rows % p.group) return hipErrorInvalidValue;
  const dim3 grid(p.rows / p.group, p.n_kv, batch), block(64 * (p.group < 4 ? p.group : 4));
  const size_t lds = (size_t)2 * nk_max * p.hd * sizeof(float);  // its keys and values, fp32
  if (dt == kBF16) {  // the attention output feeds an fp16 MFMA
    if (p.hd == 128) hipLaunchKernelGGL((merge_splits<f16, bf16, 2>), grid, block, lds, s, p);
    else hipLaunchKernelGGL((merge_splits<f16, bf16, 1>), grid, block, lds, s, p);
  } else {
    if (p.hd == 128) hipLaunchKernelGGL((merge_splits<float, float, 2>), grid, block, lds, s, p);
    else hipLaunchKernelGGL((merge_splits<float, float, 1>), grid, block, lds, s, p);
  }
  return hipGetLastError();
}

}  // namespace sp
