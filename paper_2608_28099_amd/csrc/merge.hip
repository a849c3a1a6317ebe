// Merge of the split-attention partials with the soft keys themselves
// (Sec. 3.3, Eq. 1-3).  Per query row the merge computes the soft keys visible
// to it (causal: key j' <= j) and combines them with the splits' partials
// (running max m_s in log2 units, sum l_s, unnormalised O_s) by the
// log-sum-exp rule
//   M = max(m_soft, max_s m_s),  L = l_soft 2^(m_soft-M) + sum_s l_s 2^(m_s-M),
//   O = (O_soft 2^(m_soft-M) + sum_s O_s 2^(m_s-M)) / L.
// The bf16 path's partials hold O_s / l_s in fp16 (O_s = l_s times that); the
// fp32 path's hold O_s itself.
#include "common.h"
#include "kernels.h"

namespace sp {
namespace {

// N consecutive fp32 soft operands (N a multiple of 4) with 16-byte loads.
template <int N>
__device__ __forceinline__ void soft_load_vec(const float* src, int64_t idx, float (&v)[N]) {
#pragma unroll
  for (int i = 0; i < N; i += 4) {
    const float4 x = *reinterpret_cast<const float4*>(src + idx + i);
    v[i] = x.x; v[i + 1] = x.y; v[i + 2] = x.z; v[i + 3] = x.w;
  }
}

// VALU merge (the fp32 path).  One workgroup per (sequence b, KV head g, block
// of rw consecutive soft rows with queries of one task): its rows see soft keys
// [j_lo, j] of their task (at most 64), and the workgroup stages the union,
// [j_lo, j of its last row], once in LDS (keys and values), with 16-byte loads.
// Its rw G query rows are dealt to the waves; a
// wave's first row's split partials and query are requested before the
// staging, so the two round trips overlap.  Soft scores are fp32, 16 keys per pass: lane l takes
// key j_lo + 16 ci + (l & 15) over head dims [(l >> 4) hd/4, +hd/4), and two
// shuffles add the four dim groups.  Then P V (lane l owns output dims
// l DPL .. l DPL + DPL - 1, DPL = hd / 64, each key's probability broadcast
// from its lane), and the splits folded in with a running maximum
// (log-sum-exp rule), four at a time.
template <int DPL>
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
      for (int d = 0; d < DPL; ++d) in.ov[c][d] = ((const float*)p.o_part)[row * HD + i0 + d];
    }
  };
  auto load_row = [&](int r, RowIn& in) __attribute__((always_inline)) {
    load_splits(row_base(r), 0, in);
    const int64_t qo = (((int64_t)b * p.n_kv + g) * p.r_alloc + row_qi(r) * p.group + r % p.group) * HD;
    soft_load_vec<DG>((const float*)p.q, qo + grp * DG, in.qg);
  };
  RowIn cur;
  if (wave < nrows) load_row(wave, cur);

  // stage the keys and values of the workgroup's window
  const int64_t ko = (((int64_t)b * p.n_kv + g) * p.ks + j_lo) * HD;                      // [ks][hd]
  const int64_t vo = (((p.per_seq ? (int64_t)b * p.n_kv : 0) + g) * p.ks + j_lo) * HD;  // [ks][hd]
  float* ks_ = kvs;
  float* vs_ = kvs + nk_all * HD;
  for (int e = threadIdx.x * 8; e < nk_all * HD; e += blockDim.x * 8) {
    float kx[8], vx[8];
    soft_load_vec<8>((const float*)p.k_soft, ko + e, kx);
    soft_load_vec<8>((const float*)p.v_soft, vo + e, vx);
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
    float* out = (float*)p.out + ((int64_t)b * p.out_rows + p.out_off + qi) * ((int64_t)p.n_q * HD) +
                 (int64_t)h * HD + i0;
#pragma unroll
    for (int d = 0; d < DPL; ++d) out[d] = acc[d] * inv;
  }
}

// bf16 path: the same merge with the soft-key attention on the matrix cores.
// One wave per 16-row query tile of a (sequence b, KV head g, task); the rows of
// a task are rows [task R, task R + R) of the (b, g) block, R = q_per_task group.
// Scores come transposed, S^T = K Q^T (keys along M, query rows along N), from
// bf16 hi + lo operands in three products (hi hi + hi lo + lo hi; the dropped
// lo lo term is below 2^-16 of the product), so lane l holds the scores of row
// l%16 with keys 16 kt + 4(l/16) + r.  P^T then feeds O^T = V^T P^T directly as
// the B operand: an MFMA's K index may be any fixed permutation of the keys as
// long as A uses the same one, so lane l's eight keys of a 32-key chunk are
// 4(l/16) + r and 16 + 4(l/16) + r, and the A operand reads V^T at exactly
// those keys.  V^T (hi, lo) is staged transposed in LDS once per workgroup,
// keys past the window as zeros; K and Q fragments are 16-byte loads straight
// from the soft operands.  O^T lands with lane l holding dims 16 dt + 4(l/16) + r
// of row l%16, which is also how it reads that row's split partials (16 bytes
// per dim tile) and writes its fp16 output (8 bytes).
template <int HD>
__global__ __launch_bounds__(256) void merge_soft_mfma(const MergeParams p) {
  constexpr int NC = HD / 32, NDT = HD / 16;
  extern __shared__ uint16_t vt[];  // [2][HD][ldk] bf16 bits: V^T hi, then lo
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, li = lane & 15, la = lane >> 4;
  const int g = blockIdx.y, b = blockIdx.z;
  if (p.err && *p.err) return;
  const int R = p.q_per_task * p.group;
  const int tiles = (R + 15) >> 4, wpt = (tiles + 3) >> 2;  // query tiles, workgroups per task
  const int task = blockIdx.x / wpt, t = (blockIdx.x % wpt) * 4 + wave;
  const int j_lo = task * p.k_task;
  const int nk_all = p.q_first + p.q_per_task + p.step;  // keys [j_lo, j_lo + nk_all)
  const int nkp = (nk_all + 31) & ~31, ldk = nkp + 4;

  // The lane's query fragments and the first kMl splits' (m, l) are loaded
  // before the values are staged, so their round trips overlap the staging.
  const int r = 16 * t + li;               // this lane's query row within the task (column of S^T)
  const bool valid = t < tiles && r < R;
  const int rr = valid ? r : R - 1;        // padding columns repeat the last row; never stored
  const int64_t bg = (int64_t)b * p.n_kv + g;
  const int64_t qrow = bg * p.r_alloc + (int64_t)task * R + rr;
  bf16x8 qh[NC], ql[NC];
  if (t < tiles) {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      qh[c] = __builtin_bit_cast(bf16x8, ld16v((const bf16*)p.q + qrow * HD + 32 * c + 8 * la));
      ql[c] = __builtin_bit_cast(bf16x8, ld16v((const bf16*)p.q_lo + qrow * HD + 32 * c + 8 * la));
    }
  }
  constexpr int kMl = 4;
  const int n = clamp_len(p.seq_lens, b, p.max_seq_len);
  const int ns = n > 0 ? (n + p.split_len - 1) / p.split_len : 1;
  const int64_t base = bg * p.max_splits * p.r_alloc + (int64_t)task * R + rr;
  float2 ml_pre[kMl];
#pragma unroll
  for (int sp = 0; sp < kMl; ++sp)
    if (t < tiles && sp < ns) ml_pre[sp] = p.ml_part[base + (int64_t)sp * p.r_alloc];

  // stage V^T: consecutive lanes take consecutive keys of one 8-dim chunk
  const int64_t vo = (((p.per_seq ? (int64_t)b * p.n_kv : 0) + g) * p.ks + j_lo) * HD;
  for (int e = threadIdx.x; e < nkp * (HD / 8); e += blockDim.x) {
    const int key = e % nkp, d0 = (e / nkp) * 8;
    u32x4 h = {0, 0, 0, 0}, l = {0, 0, 0, 0};
    if (key < nk_all) {
      h = ld16v((const bf16*)p.v_soft + vo + (int64_t)key * HD + d0);
      l = ld16v((const bf16*)p.v_soft_lo + vo + (int64_t)key * HD + d0);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      vt[(d0 + i) * ldk + key] = (uint16_t)(h[i >> 1] >> (16 * (i & 1)));
      vt[(HD + d0 + i) * ldk + key] = (uint16_t)(l[i >> 1] >> (16 * (i & 1)));
    }
  }
  __syncthreads();
  if (t >= tiles) return;

  const int64_t ko = (bg * p.ks + j_lo) * HD;
  const int nkt = (nk_all + 15) >> 4;
  f32x4 sc[4];
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
    sc[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (kt < nkt) {
      const int key = min(16 * kt + li, nk_all - 1);
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const bf16x8 kh = __builtin_bit_cast(bf16x8, ld16v((const bf16*)p.k_soft + ko + (int64_t)key * HD + 32 * c + 8 * la));
        const bf16x8 kl = __builtin_bit_cast(bf16x8, ld16v((const bf16*)p.k_soft_lo + ko + (int64_t)key * HD + 32 * c + 8 * la));
        sc[kt] = mfma16x16x32_bf16(kh, qh[c], sc[kt]);
        sc[kt] = mfma16x16x32_bf16(kh, ql[c], sc[kt]);
        sc[kt] = mfma16x16x32_bf16(kl, qh[c], sc[kt]);
      }
    }
  }
  // causal window of the row: keys [j_lo, j_lo + nk_r); key j_lo always visible
  const int nk_r = p.q_first + (rr / p.group) % p.q_per_task + p.step + 1;
  float M = kNegBig;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (16 * kt + 4 * la + i < nk_r) M = fmaxf(M, sc[kt][i]);
  M = fmaxf(M, __shfl_xor(M, 16));
  M = fmaxf(M, __shfl_xor(M, 32));
  float L = 0.f;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float pv = 16 * kt + 4 * la + i < nk_r ? fast_exp2(sc[kt][i] - M) : 0.f;
      sc[kt][i] = pv;
      L += pv;
    }
  L += __shfl_xor(L, 16);
  L += __shfl_xor(L, 32);

  f32x4 o[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c2 = 0; c2 < 2; ++c2) {
    if (32 * c2 < nk_all) {
      bf16x8 ph, pl;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float pv = sc[2 * c2 + (i >> 2)][i & 3];
        ph[i] = (bf16)pv;
        pl[i] = (bf16)(pv - (float)ph[i]);
      }
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const uint16_t* vr = vt + (16 * dt + li) * ldk + 32 * c2 + 4 * la;
        const u32x2 h0 = *reinterpret_cast<const u32x2*>(vr), h1 = *reinterpret_cast<const u32x2*>(vr + 16);
        const u32x2 l0 = *reinterpret_cast<const u32x2*>(vr + HD * ldk);
        const u32x2 l1 = *reinterpret_cast<const u32x2*>(vr + HD * ldk + 16);
        const bf16x8 vh = __builtin_bit_cast(bf16x8, u32x4{h0.x, h0.y, h1.x, h1.y});
        const bf16x8 vl = __builtin_bit_cast(bf16x8, u32x4{l0.x, l0.y, l1.x, l1.y});
        o[dt] = mfma16x16x32_bf16(vh, ph, o[dt]);
        o[dt] = mfma16x16x32_bf16(vh, pl, o[dt]);
        o[dt] = mfma16x16x32_bf16(vl, ph, o[dt]);
      }
    }
  }
  if (!valid) return;

  // the splits' partials, by the log-sum-exp rule (rr == r from here on)
  float Mt = M;
#pragma unroll
  for (int sp = 0; sp < kMl; ++sp)
    if (sp < ns) Mt = fmaxf(Mt, ml_pre[sp].x);
  for (int sp = kMl; sp < ns; ++sp) Mt = fmaxf(Mt, p.ml_part[base + (int64_t)sp * p.r_alloc].x);
  const float a0 = fast_exp2(M - Mt);
  L *= a0;
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) o[dt] *= a0;
  for (int sp = 0; sp < ns; ++sp) {
    const int64_t row = base + (int64_t)sp * p.r_alloc;
    float2 ml;
    if (sp < kMl) {
#pragma unroll
      for (int q = 0; q < kMl; ++q)
        if (q == sp) ml = ml_pre[q];
    } else {
      ml = p.ml_part[row];
    }
    const float w = ml.y * fast_exp2(ml.x - Mt);  // the partial is O_s / l_s
    L += w;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      const f16x4 v = *reinterpret_cast<const f16x4*>((const f16*)p.o_part + row * HD + 16 * dt + 4 * la);
      o[dt] += f32x4{(float)v[0], (float)v[1], (float)v[2], (float)v[3]} * w;
    }
  }
  const float inv = 1.0f / L;
  const int qi = task * p.q_per_task + r / p.group, h = g * p.group + r % p.group;
  f16* out = (f16*)p.out + ((int64_t)b * p.out_rows + p.out_off + qi) * ((int64_t)p.n_q * HD) + (int64_t)h * HD + 4 * la;
  bool oor = false;
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) {
    f16x4 y;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float v = o[dt][i] * inv;
      oor |= !(fabsf(v) <= 65504.0f);
      y[i] = (f16)v;
    }
    *reinterpret_cast<f16x4*>(out + 16 * dt) = y;
  }
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
  // bf16 storage: matrix-core merge, up to four query tiles per workgroup (one
  // per wave), fp16 output for the o-projection's fp16 MFMA.  Against the
  // VALU merge below on the same rows: 27B shape 0.15 ms against 0.39 ms, the
  // ragged 9B shape 31 us against 65 us.
  if (dt == kBF16) {
    const int R = p.q_per_task * p.group, tiles = (R + 15) / 16;
    const int nkp = (nk_max + 31) & ~31;
    const dim3 grid(tasks * ((tiles + 3) / 4), p.n_kv, batch), block(64 * (tiles < 4 ? tiles : 4));
    const size_t lds = (size_t)2 * p.hd * (nkp + 4) * sizeof(uint16_t);
    if (p.hd == 128) hipLaunchKernelGGL(merge_soft_mfma<128>, grid, block, lds, s, p);
    else hipLaunchKernelGGL(merge_soft_mfma<64>, grid, block, lds, s, p);
    return hipGetLastError();
  }
  // fp32 path.  Soft rows per workgroup: the most (a power of two) that still
  // leave min_wgs workgroups (4 per compute unit).  Each workgroup stages its
  // key window once and then streams its rows' partials.
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
  if (p.hd == 128) hipLaunchKernelGGL(merge_splits<2>, grid, block, lds, s, q);
  else hipLaunchKernelGGL(merge_splits<1>, grid, block, lds, s, q);
  return hipGetLastError();
}

}  // namespace sp
