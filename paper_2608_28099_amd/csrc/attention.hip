// Split attention of the k soft queries over the cached prefix plus the soft
// keys (Sec. 3.3 Eq. 1-3), and the merge of the splits.
//
// Work unit: one wave per (sequence b, KV head g, query group, split s).  The
// rows of a KV head are its k*G soft queries (row r = j*G + h%G for soft row j
// and query head h = g*G + h%G); a query group is 16*QT consecutive rows.
// Split s covers cache tokens [s*split_len, min(N_b, (s+1)*split_len)); split 0
// also covers the soft keys.  Each wave keeps an online softmax (running max m
// in log2 units, running sum l, unnormalised output O) and writes them as a
// partial; the merge combines partials with the log-sum-exp rule
//   M = max_s m_s,  L = sum_s l_s 2^(m_s - M),  O = sum_s O_s 2^(m_s - M) / L.
//
// bf16 path (bf16 KV cache, fp16 MFMA operands, fp32 accumulation), per
// 16-token chunk (always inside one block, so one block-table lookup per chunk,
// uniform across the wave):
//   S^T = K Q^T on v_mfma_f32_16x16x32_f16 with the 16 tokens as MFMA rows:
//   lane (li, la) loads K row li (16-byte pieces of the chunked K tile) and,
//   after the MFMA, holds the scores of tokens 4la .. 4la+3 for query li.  That
//   is exactly the A operand of v_mfma_f32_16x16x16_f16 (query row li, 4
//   consecutive tokens), so P never goes through LDS.
//   O += P V with V as the B operand: lane (li, la) needs V[4la .. 4la+3][16nt + li],
//   one 8-byte load from the dim-major V tile; the 16 lanes of a row read 512
//   contiguous bytes.  K and V are loaded as bf16 with streaming loads and
//   converted to fp16 in registers (exact for |x| in [2^-14, 65504]); the queries
//   and the soft rows' K/V arrive in fp16.
//   All query tiles' QK products are issued before any softmax work, and one
//   wave-wide test per chunk decides whether a reference max must move, so the
//   common path is one basic block the scheduler can overlap.
#include "common.h"
#include "kernels.h"

#ifndef SP_ATTN_DEPTH
#define SP_ATTN_DEPTH 3
#endif

namespace sp {
namespace {

__device__ __forceinline__ int clamp_len(const int* seq_lens, int b, int max_seq_len) {
  int n = seq_lens[b];
  return n < 0 ? 0 : (n > max_seq_len ? max_seq_len : n);
}

__device__ __forceinline__ int64_t phys_block(const AttnParams& p, int b, int t) {
  const int lb = t >> p.bs_log2;
  return p.block_table ? (int64_t)p.block_table[(int64_t)b * p.mbps + lb]
                       : (int64_t)b * p.mbps + lb;
}

template <int HD>
struct Frag {
  static constexpr int NC = HD / 32;  // 32-wide head-dim chunks (QK contraction)
  static constexpr int NT = HD / 16;  // 16-wide head-dim tiles (PV output)
  uint4 k[NC];                        // K[token li][8 (la*NC + c) .. +7]
  uint2 v[NT];                        // V[tokens 4la .. 4la+3][16nt + li]
};

// kt/vt: K and V tile bases of the block holding the chunk, slot0: slot of the
// chunk's first token in that block, bs: tile length in tokens.  STREAM: the
// KV cache, read once (non-temporal loads).
template <int HD, bool STREAM, typename T>
__device__ __forceinline__ void load_frag(Frag<HD>& f, const T* kt, const T* vt, int slot0, int bs,
                                          int li, int la) {
  constexpr int NC = Frag<HD>::NC, NT = Frag<HD>::NT;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const T* a = kt + ((int64_t)(la * NC + c) * bs + slot0 + li) * 8;
    f.k[c] = STREAM ? ld16_stream(a) : ld16(a);
  }
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const T* a = vt + (int64_t)(16 * nt + li) * bs + slot0 + 4 * la;
    f.v[nt] = STREAM ? ld8_stream(a) : *reinterpret_cast<const uint2*>(a);
  }
}

enum { kFull = 0, kTail = 1, kSoft = 2 };

// A row's reference max moves only when a score exceeds it by more than this
// (log2 units), so probabilities stay below 2^8 between moves.
constexpr float kRescaleLog2 = 8.0f;

// One 16-token chunk.  limit: tokens of the chunk that are data (kTail);
// key0, row0, group, k: soft-key causal mask (kSoft).  Cache chunks hold bf16
// (converted here), the soft chunk fp16.
template <int HD, int QT, int MODE>
__device__ __forceinline__ void process_chunk(Frag<HD>& f, const f16x8 (&qf)[QT][HD / 32],
                                              f32x4 (&o)[QT][HD / 16], float (&m)[QT],
                                              float (&l)[QT], int li, int la, int limit,
                                              int key0, int row0, int group, int k) {
  constexpr int NC = HD / 32, NT = HD / 16;
  if (MODE != kSoft) {
#pragma unroll
    for (int c = 0; c < NC; ++c) f.k[c] = bf16x8_to_f16x8(f.k[c]);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) f.v[nt] = bf16x4_to_f16x4(f.v[nt]);
  }
  if (MODE == kTail) {
    // Tokens at or past `limit` carry arbitrary bytes (NaN poison included):
    // their V entries are replaced by 0 and their scores by -inf.
    const int keep = limit - 4 * la;  // tokens of this lane kept: 4la + r < limit
    const uint32_t lo = keep >= 2 ? 0xffffffffu : (keep == 1 ? 0x0000ffffu : 0u);
    const uint32_t hi = keep >= 4 ? 0xffffffffu : (keep == 3 ? 0x0000ffffu : 0u);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      f.v[nt].x &= lo;
      f.v[nt].y &= hi;
    }
  }
  // scores: st[qt][r] is token 4la + r of the chunk, query li of tile qt
  f32x4 st[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) st[qt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) st[qt] = mfma16x16x32(as_f16x8(f.k[c]), qf[qt][c], st[qt]);
  bool move = false;
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    if (MODE == kTail) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (4 * la + r >= limit) st[qt][r] = -INFINITY;
    } else if (MODE == kSoft) {
      // soft key j' is visible to query row r iff j' <= r / G (causal, own row included)
      int jmax = (row0 + 16 * qt + li) / group;
      jmax = jmax < k - 1 ? jmax : k - 1;
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (key0 + 4 * la + r > jmax) st[qt][r] = -INFINITY;
    }
    const float lmax = fmaxf(fmaxf(st[qt][0], st[qt][1]), fmaxf(st[qt][2], st[qt][3]));
    move |= lmax > m[qt] + kRescaleLog2;
  }
  // Lazy reference max: p = 2^(s - m) with m the row's reference, which only
  // moves (with the cross-lane reduction and the rescale of l and O) when some
  // score exceeds it by more than kRescaleLog2.
  if (__any(move)) {
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      float lmax = fmaxf(fmaxf(st[qt][0], st[qt][1]), fmaxf(st[qt][2], st[qt][3]));
      lmax = fmaxf(lmax, __shfl_xor(lmax, 16));
      lmax = fmaxf(lmax, __shfl_xor(lmax, 32));
      const float mn = fmaxf(m[qt], lmax);
      const float alpha = fast_exp2(m[qt] - mn);
      l[qt] *= alpha;
      m[qt] = mn;
      // O rows held by this lane are queries 4la + r; their factors live in lanes 4la + r.
      float ar[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) ar[r] = __shfl(alpha, 4 * la + r);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int r = 0; r < 4; ++r) o[qt][nt][r] *= ar[r];
    }
  }
  f16x4 pa[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    float ps = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float pv = fast_exp2(st[qt][r] - m[qt]);
      ps += pv;
      pa[qt][r] = (f16)pv;
    }
    l[qt] += ps;
  }
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) o[qt][nt] = mfma16x16x16(pa[qt], as_f16x4(f.v[nt]), o[qt][nt]);
}

// DEPTH fragment buffers rotate: while chunk i runs, chunks i+1 .. i+DEPTH-1 are
// in flight.
template <int HD, int QT, int DEPTH>
__global__ __launch_bounds__(64) void attn_split_bf16(const AttnParams p) {
  constexpr int NC = HD / 32, NT = HD / 16;
  const int lane = threadIdx.x, li = lane & 15, la = lane >> 4;
  const int s = blockIdx.x;
  const int g = blockIdx.y / p.n_qgroups, qg = blockIdx.y % p.n_qgroups;
  const int b = blockIdx.z;
  if (p.err && *p.err) return;
  const int n = clamp_len(p.seq_lens, b, p.max_seq_len);
  const int t0 = s * p.split_len;
  if (s > 0 && t0 >= n) return;
  const int t1 = min(n, t0 + p.split_len);
  const int row0 = qg * 16 * QT;
  const int bs = 1 << p.bs_log2;

  const f16* qb = (const f16*)p.q + (((int64_t)b * p.n_kv + g) * p.r_alloc + row0) * HD;
  f16x8 qf[QT][NC];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt)
#pragma unroll
    for (int c = 0; c < NC; ++c)
      qf[qt][c] = as_f16x8(ld16(qb + (int64_t)(16 * qt + li) * HD + 8 * (la * NC + c)));

  f32x4 o[QT][NT];
  float m[QT], l[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    m[qt] = kNegBig;
    l[qt] = 0.f;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) o[qt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  if (s == 0) {
    const f16* kt = (const f16*)p.k_soft + ((int64_t)b * p.n_kv + g) * p.ks * HD;
    const f16* vt = (const f16*)p.v_soft + (int64_t)g * HD * p.ks;
    for (int c0 = 0; c0 < p.k; c0 += 16) {
      Frag<HD> f;
      load_frag<HD, false>(f, kt, vt, c0, p.ks, li, la);
      process_chunk<HD, QT, kSoft>(f, qf, o, m, l, li, la, 0, c0, row0, p.group, p.k);
    }
  }

  if (t0 < t1) {
    const bf16* kbase = (const bf16*)p.k_base + (int64_t)g * p.k_sh;
    const bf16* vbase = (const bf16*)p.v_base + (int64_t)g * p.v_sh;
    // A 16-token chunk starting at a multiple of 16 lies inside one block, and
    // its first token is valid, so the block is one the sequence owns.
    auto load_cache = [&](Frag<HD>& f, int c0) {
      const int64_t blk = phys_block(p, b, c0);
      load_frag<HD, true>(f, kbase + blk * p.k_sb, vbase + blk * p.v_sb, c0 & (bs - 1), bs, li, la);
    };
    // Prefetch addresses are clamped to the last full chunk, so every load
    // stays inside the sequence.
    const int nfull = (t1 - t0) >> 4, rem = (t1 - t0) & 15;
    Frag<HD> buf[DEPTH];
    if (nfull > 0) {
#pragma unroll
      for (int j = 0; j < DEPTH - 1; ++j) load_cache(buf[j], t0 + 16 * (j < nfull ? j : nfull - 1));
    }
    for (int i = 0; i < nfull; i += DEPTH) {
#pragma unroll
      for (int u = 0; u < DEPTH; ++u) {
        if (i + u < nfull) {
          const int nx = i + u + DEPTH - 1;
          load_cache(buf[(u + DEPTH - 1) % DEPTH], t0 + 16 * (nx < nfull ? nx : nfull - 1));
          process_chunk<HD, QT, kFull>(buf[u], qf, o, m, l, li, la, 16, 0, row0, p.group, p.k);
        }
      }
    }
    if (rem) {
      Frag<HD> f;
      load_cache(f, t0 + 16 * nfull);
      process_chunk<HD, QT, kTail>(f, qf, o, m, l, li, la, rem, 0, row0, p.group, p.k);
    }
  }

  const int64_t prow = (((int64_t)b * p.n_kv + g) * p.max_splits + s) * p.r_alloc + row0;
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    float lt = l[qt];
    lt += __shfl_xor(lt, 16);
    lt += __shfl_xor(lt, 32);
    if (la == 0) p.ml_part[prow + 16 * qt + li] = make_float2(m[qt], lt);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        p.o_part[(prow + 16 * qt + 4 * la + r) * HD + 16 * nt + li] = o[qt][nt][r];
  }
}

// ---------------------------------------------------------------- fp32 path
// One workgroup (256 threads) per (b, g, split), all rows (<= 64) of the KV
// head; K/V tiles of 32 tokens staged in LDS, plain fp32 arithmetic.
template <int HD>
__global__ __launch_bounds__(256) void attn_split_f32(const AttnParams p) {
  constexpr int TT = 32, X = 4;
  constexpr int OPT = 64 * HD / 256;  // output elements per thread (max rows 64)
  __shared__ float qs[64][HD + 1];
  __shared__ float ks[TT][HD + 1];
  __shared__ float vs[TT][HD + 1];
  __shared__ float ps[64][TT + 1];
  __shared__ float alpha_s[64], m_s[64], l_s[64];
  const int tid = threadIdx.x;
  const int s = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  if (p.err && *p.err) return;
  const int n = clamp_len(p.seq_lens, b, p.max_seq_len);
  const int t0 = s * p.split_len;
  if (s > 0 && t0 >= n) return;
  const int t1 = min(n, t0 + p.split_len);
  const int R = p.rows;
  const int bs = 1 << p.bs_log2;

  const float* qb = (const float*)p.q + ((int64_t)b * p.n_kv + g) * p.r_alloc * HD;
  for (int idx = tid; idx < R * HD; idx += 256) qs[idx / HD][idx % HD] = qb[idx];
  if (tid < 64) {
    m_s[tid] = kNegBig;
    l_s[tid] = 0.f;
  }
  float oacc[OPT];
#pragma unroll
  for (int u = 0; u < OPT; ++u) oacc[u] = 0.f;
  __syncthreads();

  // is_soft: chunk of soft keys starting at key c0; else cache tokens [c0, c0 + TT).
  auto run_chunk = [&](bool is_soft, int c0) {
    for (int idx = tid; idx < TT * HD; idx += 256) {
      const int t = idx / HD, i = idx % HD, tok = c0 + t;
      float kv = 0.f, vv = 0.f;
      if (is_soft) {
        if (tok < p.k) {
          const float* kt = (const float*)p.k_soft + ((int64_t)b * p.n_kv + g) * p.ks * HD;
          const float* vt = (const float*)p.v_soft + (int64_t)g * HD * p.ks;
          kv = kt[((int64_t)(i / X) * p.ks + tok) * X + i % X];
          vv = vt[(int64_t)i * p.ks + tok];
        }
      } else if (tok < t1) {
        const int64_t blk = phys_block(p, b, tok);
        const int slot = tok & (bs - 1);
        const float* kt = (const float*)p.k_base + blk * p.k_sb + (int64_t)g * p.k_sh;
        const float* vt = (const float*)p.v_base + blk * p.v_sb + (int64_t)g * p.v_sh;
        kv = kt[((int64_t)(i / X) * bs + slot) * X + i % X];
        vv = vt[(int64_t)i * bs + slot];
      }
      ks[t][i] = kv;
      vs[t][i] = vv;
    }
    __syncthreads();
    for (int idx = tid; idx < R * TT; idx += 256) {
      const int r = idx / TT, t = idx % TT, tok = c0 + t;
      float acc = 0.f;
      for (int i = 0; i < HD; ++i) acc += qs[r][i] * ks[t][i];
      bool ok;
      if (is_soft) {
        int jmax = r / p.group;
        jmax = jmax < p.k - 1 ? jmax : p.k - 1;
        ok = tok <= jmax;
      } else {
        ok = tok < t1;
      }
      ps[r][t] = ok ? acc : -INFINITY;
    }
    __syncthreads();
    if (tid < R) {
      float mx = m_s[tid];
      for (int t = 0; t < TT; ++t) mx = fmaxf(mx, ps[tid][t]);
      const float a = exp2f(m_s[tid] - mx);
      float sum = 0.f;
      for (int t = 0; t < TT; ++t) {
        const float e = exp2f(ps[tid][t] - mx);
        ps[tid][t] = e;
        sum += e;
      }
      l_s[tid] = l_s[tid] * a + sum;
      m_s[tid] = mx;
      alpha_s[tid] = a;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < OPT; ++u) {
      const int idx = tid + 256 * u;
      const int r = idx / HD, i = idx % HD;
      if (r < R) {
        float acc = oacc[u] * alpha_s[r];
        for (int t = 0; t < TT; ++t) acc += ps[r][t] * vs[t][i];
        oacc[u] = acc;
      }
    }
    __syncthreads();
  };

  if (s == 0)
    for (int c0 = 0; c0 < p.k; c0 += TT) run_chunk(true, c0);
  for (int c0 = t0; c0 < t1; c0 += TT) run_chunk(false, c0);

  const int64_t prow = (((int64_t)b * p.n_kv + g) * p.max_splits + s) * p.r_alloc;
  if (tid < R) p.ml_part[prow + tid] = make_float2(m_s[tid], l_s[tid]);
#pragma unroll
  for (int u = 0; u < OPT; ++u) {
    const int idx = tid + 256 * u;
    const int r = idx / HD, i = idx % HD;
    if (r < R) p.o_part[(prow + r) * HD + i] = oacc[u];
  }
}

// ---------------------------------------------------------------- merge
// One wave per row (b, g, r); lanes cover the head dimension.
template <typename T>
__global__ __launch_bounds__(256) void merge_splits(const MergeParams p) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + wave, g = blockIdx.y, b = blockIdx.z;
  if (r >= p.rows) return;
  if (p.err && *p.err) return;
  const int n = clamp_len(p.seq_lens, b, p.max_seq_len);
  const int ns = n > 0 ? (n + p.split_len - 1) / p.split_len : 1;
  const int64_t base = ((int64_t)b * p.n_kv + g) * p.max_splits * p.r_alloc + r;
  float M = kNegBig;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, p.ml_part[base + (int64_t)s * p.r_alloc].x);
  float L = 0.f;
  for (int s = 0; s < ns; ++s) {
    const float2 ml = p.ml_part[base + (int64_t)s * p.r_alloc];
    L += ml.y * fast_exp2(ml.x - M);
  }
  const float inv = 1.0f / L;
  const int j = r / p.group, h = g * p.group + r % p.group;
  T* out = (T*)p.out + ((int64_t)b * p.k + j) * ((int64_t)p.n_q * p.hd) + (int64_t)h * p.hd;
  for (int i = lane; i < p.hd; i += 64) {
    float acc = 0.f;
    for (int s = 0; s < ns; ++s) {
      const int64_t row = base + (int64_t)s * p.r_alloc;
      acc += p.o_part[row * p.hd + i] * fast_exp2(p.ml_part[row].x - M);
    }
    out[i] = from_f32<T>(acc * inv);
  }
}

}  // namespace

// Prefetch depth of the production instantiation.
constexpr int kAttnDepth = SP_ATTN_DEPTH;

hipError_t launch_attention_bf16(const AttnParams& p, int hd, int qt, int batch, hipStream_t s) {
  const dim3 grid(p.max_splits, p.n_kv * p.n_qgroups, batch);
#define SP_ATTN_CASE(HD_, QT_)                                                                  \
  if (hd == HD_ && qt == QT_) {                                                                 \
    hipLaunchKernelGGL((attn_split_bf16<HD_, QT_, kAttnDepth>), grid, dim3(64), 0, s, p);  \
    return hipGetLastError();                                                                   \
  }
  SP_ATTN_CASE(128, 1) SP_ATTN_CASE(128, 2) SP_ATTN_CASE(128, 3) SP_ATTN_CASE(128, 4)
  SP_ATTN_CASE(64, 1) SP_ATTN_CASE(64, 2) SP_ATTN_CASE(64, 3) SP_ATTN_CASE(64, 4)
  SP_ATTN_CASE(64, 5)
#undef SP_ATTN_CASE
  return hipErrorInvalidValue;
}

hipError_t launch_attention_f32(const AttnParams& p, int hd, int batch, hipStream_t s) {
  const dim3 grid(p.max_splits, p.n_kv, batch);
  if (hd == 128)
    hipLaunchKernelGGL(attn_split_f32<128>, grid, dim3(256), 0, s, p);
  else if (hd == 64)
    hipLaunchKernelGGL(attn_split_f32<64>, grid, dim3(256), 0, s, p);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_merge(DType dt, const MergeParams& p, int batch, hipStream_t s) {
  const dim3 grid((p.rows + 3) / 4, p.n_kv, batch);
  if (dt == kBF16)  // the attention output feeds an fp16 MFMA
    hipLaunchKernelGGL(merge_splits<f16>, grid, dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL(merge_splits<float>, grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace sp
