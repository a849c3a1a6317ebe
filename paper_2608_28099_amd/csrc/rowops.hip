// Row kernels of the probe forward: RMSNorm, RoPE at positions N_b + j with the
// scatter into the attention layouts, final norm + read-out + linear
// classifier, and the debug validation of device-resident metadata.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace sp {
namespace {

// ---------------------------------------------------------------- RMSNorm
// One workgroup (256 threads) per row; the row is read once, 4 values per
// load, and kept in registers between the sum of squares and the scaling
// (d <= 256 * 4 * kRowChunks = 16384, d % 4 == 0).
constexpr int kRowChunks = 16;

template <typename T>
__device__ __forceinline__ void load4(const T* p, float (&v)[4]) {
  if constexpr (sizeof(T) == 4) {
    const float4 x = *reinterpret_cast<const float4*>(p);
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
  } else {
    const uint2 x = *reinterpret_cast<const uint2*>(p);
    const T* h = reinterpret_cast<const T*>(&x);
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = to_f32(h[e]);
  }
}
template <typename T>
__device__ __forceinline__ void store4(T* p, const float (&v)[4]) {
  if constexpr (sizeof(T) == 4) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  } else {
    T h[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) h[e] = from_f32<T>(v[e]);
    *reinterpret_cast<uint2*>(p) = *reinterpret_cast<const uint2*>(h);
  }
}

// Sets kStatusRange in *status (nullable) when an fp16 output leaves fp16's
// range (it is then stored as inf).
__device__ __forceinline__ void flag_range(bool out_of_range, int* status) {
  if (__any(out_of_range) && (threadIdx.x & 63) == 0 && status) atomicOr(status, kStatusRange);
}

// CH: chunks of 1024 values held per row (registers scale with it, so the
// launcher takes the fewest that cover d).
template <typename TI, typename TG, typename TO, int CH>
__global__ __launch_bounds__(256) void rmsnorm_rows(const TI* x, int64_t ld_x, const TG* gain,
                                                    const TG* gain2, TO* out, int64_t ld_out, int d,
                                                    float eps, int* status) {
  constexpr int kRowChunks = CH;
  __shared__ float red[4];
  const int r = blockIdx.x;
  const TI* xr = x + (int64_t)r * ld_x;
  float v[kRowChunks][4], gv[kRowChunks][4];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < kRowChunks; ++c) {
    const int i = 4 * (threadIdx.x + 256 * c);
    if (i < d) load4(xr + i, v[c]);
  }
  // the gains are loaded under the row's loads and reduction (one round trip, not two)
#pragma unroll
  for (int c = 0; c < kRowChunks; ++c) {
    const int i = 4 * (threadIdx.x + 256 * c);
    if (i < d) load4(gain + i, gv[c]);
  }
#pragma unroll
  for (int c = 0; c < kRowChunks; ++c) {
    const int i = 4 * (threadIdx.x + 256 * c);
    if (i < d) {
#pragma unroll
      for (int e = 0; e < 4; ++e) ss += v[c][e] * v[c][e];
    }
  }
  ss = block_sum_256(ss, red);
  float inv = 1.0f / sqrtf(ss / (float)d + eps);
  // optional second norm of the result with gain2 (two RMSNorms in a row)
  for (int pass = 0; pass < (gain2 ? 2 : 1); ++pass) {
    float ss2 = 0.f;
#pragma unroll
    for (int c = 0; c < kRowChunks; ++c) {
      const int i = 4 * (threadIdx.x + 256 * c);
      if (i < d) {
        if (pass) load4(gain2 + i, gv[c]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[c][e] = v[c][e] * inv * gv[c][e];
          ss2 += v[c][e] * v[c][e];
        }
      }
    }
    if (gain2 && pass == 0) {
      ss2 = block_sum_256(ss2, red);
      inv = 1.0f / sqrtf(ss2 / (float)d + eps);
    }
  }
  TO* orow = out + (int64_t)r * ld_out;
  bool oor = false;
#pragma unroll
  for (int c = 0; c < kRowChunks; ++c) {
    const int i = 4 * (threadIdx.x + 256 * c);
    if (i < d) {
      store4(orow + i, v[c]);
      if constexpr (sizeof(TO) == 2)
#pragma unroll
        for (int e = 0; e < 4; ++e) oor |= !(fabsf(v[c][e]) <= 65504.0f);
    }
  }
  if constexpr (sizeof(TO) == 2) flag_range(oor, status);
}

// ---------------------------------------------------------------- RoPE + scatter
// One workgroup per (block of up to kRopeRows soft rows j, sequence b): the
// rotation of pair (i, i + hd/2) at row j's position N_b + t (t = step +
// j % k_task) by angle (N_b + t) * base^(-2i/hd) is computed once per row, in
// fp64, into LDS, then applied to the row's key heads (soft slot step + j)
// and, for rows that carry queries, its query heads, two adjacent pairs per
// lane (4-byte stores of bf16 pairs, 8-byte of fp32).  The value heads are not
// rotated; in the one-pass form (per_seq = 0) they are the same for every
// sequence and written by b = 0, in the recursive form every sequence has its
// own row of projections ([B][k] rows) and its own values.  Rows per
// workgroup: as many as keep two workgroups per compute unit (one row each
// made the 27B-shaped batch 8192 workgroups with a few hundred stores each:
// 69-76 us, the same with the trigonometry taken out).
// SPLIT (T = bf16): each value x is stored as hi = bf16(x) and lo = bf16(x - hi).
constexpr int kRopeRows = 8;

template <typename T, bool SPLIT>
__device__ __forceinline__ void put2(void* hi, void* lo, int64_t idx, float x0, float x1) {  // idx even
  if constexpr (sizeof(T) == 2) {
    const T h0 = from_f32<T>(x0), h1 = from_f32<T>(x1);
    auto pack = [](T a, T b) {
      return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
    };
    *(uint32_t*)((T*)hi + idx) = pack(h0, h1);
    if (SPLIT) *(uint32_t*)((T*)lo + idx) = pack(from_f32<T>(x0 - to_f32(h0)), from_f32<T>(x1 - to_f32(h1)));
  } else {
    static_assert(!SPLIT, "fp32 values are stored whole");
    *(float2*)((T*)hi + idx) = make_float2(x0, x1);
  }
}

template <typename T, bool SPLIT>
__global__ __launch_bounds__(256) void rope_scatter(const RopeParams p, int rows_per_block) {
  __shared__ float cs[kRopeRows][64], sn[kRopeRows][64];  // hd / 2 <= 64
  const int b = blockIdx.y, j0 = blockIdx.x * rows_per_block;
  if (p.err && *p.err) return;
  const int hd = p.hd, half = hd / 2, hp = half / 2;  // hp: lanes per head (two pairs each)
  const int nj = min(rows_per_block, p.k - j0);
  int n = p.seq_lens[b];
  // a length outside [0, max_seq_len] is clamped (every kernel does the same)
  // and reported through the status word
  if ((n < 0 || n > p.max_seq_len) && blockIdx.x == 0 && threadIdx.x == 0 && p.status)
    atomicOr(p.status, kStatusSeqLen);
  n = n < 0 ? 0 : (n > p.max_seq_len ? p.max_seq_len : n);
  for (int t = threadIdx.x; t < nj * half; t += blockDim.x) {
    const int jr = t / half, i = t % half;
    const int jj = (j0 + jr) % p.k_task;
    const double theta = pow(p.rope_base, -2.0 * (double)i / (double)hd);
    const double ang = (double)(n + p.step + jj) * theta;
    cs[jr][i] = (float)cos(ang);
    sn[jr][i] = (float)sin(ang);
  }
  __syncthreads();
  const int nh = p.n_q + p.n_kv;
  for (int jr = 0; jr < nj; ++jr) {
    const int j = j0 + jr, jj = j % p.k_task, slot = p.step + j;
    const float* row = p.qkv + ((int64_t)(p.per_seq ? b * p.k : 0) + j) * (p.n_q + 2 * p.n_kv) * hd;
    const int qi = (j / p.k_task) * p.q_per_task + jj - p.q_first;
    for (int e = (jj >= p.q_first ? 0 : p.n_q * hp) + threadIdx.x; e < nh * hp; e += blockDim.x) {
      const int h = e / hp, i = 2 * (e % hp);
      const float2 xa = *(const float2*)(row + h * hd + i), xb = *(const float2*)(row + h * hd + i + half);
      const float c0 = cs[jr][i], s0 = sn[jr][i], c1 = cs[jr][i + 1], s1 = sn[jr][i + 1];
      const float r0a = xa.x * c0 - xb.x * s0, r1a = xb.x * c0 + xa.x * s0;
      const float r0b = xa.y * c1 - xb.y * s1, r1b = xb.y * c1 + xa.y * s1;
      if (h < p.n_q) {
        const int g = h / p.group, rr = qi * p.group + h % p.group;
        const int64_t base = (((int64_t)b * p.n_kv + g) * p.r_alloc + rr) * hd;
        put2<T, SPLIT>(p.q, p.q_lo, base + i, r0a * p.q_scale, r0b * p.q_scale);
        put2<T, SPLIT>(p.q, p.q_lo, base + i + half, r1a * p.q_scale, r1b * p.q_scale);
      } else {
        const int g = h - p.n_q;
        const int64_t base = (((int64_t)b * p.n_kv + g) * p.ks + slot) * hd;
        put2<T, SPLIT>(p.k_soft, p.k_soft_lo, base + i, r0a, r0b);
        put2<T, SPLIT>(p.k_soft, p.k_soft_lo, base + i + half, r1a, r1b);
      }
    }
    if (p.per_seq || b == 0) {
      const int64_t vb = p.per_seq ? (int64_t)b * p.n_kv : 0;
      for (int e = threadIdx.x; e < p.n_kv * half; e += blockDim.x) {
        const int g = e / half, i = 2 * (e % half);
        const float2 v = *(const float2*)(row + (p.n_q + p.n_kv + g) * hd + i);
        put2<T, SPLIT>(p.v_soft, p.v_soft_lo, ((vb + g) * p.ks + slot) * hd + i, v.x, v.y);
      }
    }
  }
}

// ---------------------------------------------------------------- read-out
// One workgroup per (sequence b, task t, class c):
//   logits[b][t][c] = sum_j w_j * inv_j * sum_i W_cls[t][c][i] gamma_i y_j[i]  (+ bias[t][c]),
// with inv_j = 1 / sqrt(mean_i y_j[i]^2 + eps) over the read-out rows j of task
// t (its last row, w = 1; or all k, w = 1/k): RMSNorm, pooling and the linear
// classifier folded into one pass and one block reduction per row.
template <typename T>
__global__ __launch_bounds__(256) void final_classifier(const ClsParams p) {
  __shared__ float red[4];
  const int b = blockIdx.x, tc = blockIdx.y, d = p.d;  // tc = task * C + class
  if (p.err && *p.err) return;
  const int task = tc / p.n_classes;
  const int j0 = p.pool_mean ? 0 : p.k - 1;
  const float w = p.pool_mean ? 1.0f / (float)p.k : 1.0f;
  const T* wr = (const T*)p.w_cls + (p.cls_rows ? (int64_t)p.cls_rows[tc] : (int64_t)tc) * d;
  const T* gm = (const T*)p.final_norm;
  float wg[kRowChunks][4];  // W_cls[c][i] * gamma_i, reused for every row
#pragma unroll
  for (int q = 0; q < kRowChunks; ++q) {
    const int i = 4 * (threadIdx.x + 256 * q);
    if (i < d) {
      float a[4], g4[4];
      load4(wr + i, a);
      load4(gm + i, g4);
#pragma unroll
      for (int e = 0; e < 4; ++e) wg[q][e] = a[e] * g4[e];
    }
  }
  float logit = 0.f;
  for (int j = j0; j < p.k; ++j) {
    const float* yr = p.y + (((int64_t)b * p.n_tasks + task) * p.k + j) * d;
    float ss = 0.f, dot = 0.f;
#pragma unroll
    for (int q = 0; q < kRowChunks; ++q) {
      const int i = 4 * (threadIdx.x + 256 * q);
      if (i < d) {
        float y4[4];
        load4(yr + i, y4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          ss += y4[e] * y4[e];
          dot += y4[e] * wg[q][e];
        }
      }
    }
    ss = block_sum_256(ss, red);
    dot = block_sum_256(dot, red);
    logit += w * dot / sqrtf(ss / (float)d + p.eps);
  }
  if (threadIdx.x == 0)
    p.logits[(int64_t)b * p.n_tasks * p.n_classes + tc] = logit + (p.b_cls ? p.b_cls[tc] : 0.f);
}

// ---------------------------------------------------------------- fp16 staging with row scales
// One workgroup per row: max |x| over the row, then the scaled fp16 copy.
__global__ __launch_bounds__(256) void scale_rows_f16(const bf16* x, int64_t ld_x, f16* out,
                                                      float* inv_scale, int cols) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  const bf16* xr = x + (int64_t)r * ld_x;
  float mx = 0.f;
  for (int i = threadIdx.x; i < cols; i += 256) mx = fmaxf(mx, fabsf(to_f32(xr[i])));
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  int e = 0;
  while (e < 126 && ldexpf(mx, -e) >= 32768.0f) ++e;
  const float sc = ldexpf(1.0f, -e);
  f16* orow = out + (int64_t)r * cols;
  for (int i = threadIdx.x; i < cols; i += 256) orow[i] = (f16)(to_f32(xr[i]) * sc);
  if (threadIdx.x == 0) inv_scale[r] = ldexpf(1.0f, e);
}

// ---------------------------------------------------------------- validation
__global__ void validate_meta(const ValidateParams p) {
  const int b = blockIdx.x;
  if (b == 0 && p.cls_rows) {
    for (int i = threadIdx.x; i < p.n_cls_rows; i += blockDim.x) {
      const int r = p.cls_rows[i];
      if (r < 0 || (int64_t)r >= p.cls_vocab) atomicOr(p.err, 8);
    }
  }
  const int n = p.seq_lens[b];
  if (n < 0 || n > p.max_seq_len) {
    if (threadIdx.x == 0) atomicOr(p.err, 1);
    return;
  }
  const int nblk = (n + (1 << p.bs_log2) - 1) >> p.bs_log2;
  if (nblk > p.mbps) {
    if (threadIdx.x == 0) atomicOr(p.err, 2);
    return;
  }
  if (!p.block_table) return;
  for (int j = threadIdx.x; j < nblk; j += blockDim.x) {
    const int id = p.block_table[(int64_t)b * p.mbps + j];
    if (id < 0 || (int64_t)id >= p.num_blocks) atomicOr(p.err, 4);
  }
}

// ---------------------------------------------------------------- workspace guards, weight image
__global__ void fill_words(uint32_t* p, size_t n, uint32_t value) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = value;
}

// One workgroup per guard area.
__global__ void check_guards(const char* base, const uint64_t* offs, int words, uint32_t value, int* flag,
                             int bit) {
  const uint32_t* g = reinterpret_cast<const uint32_t*>(base + offs[blockIdx.x]);
  bool bad = false;
  for (int i = threadIdx.x; i < words; i += blockDim.x) bad |= g[i] != value;
  if (__any(bad) && (threadIdx.x & 63) == 0) atomicOr(flag, bit);
}

__global__ void bf16_to_f16(const uint32_t* src, uint32_t* dst, size_t n2) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n2; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = bf16x2_to_f16x2(src[i]);
}

__global__ void check_header(const uint32_t* image, const uint32_t* expect, int n_words, int* flag, int bit) {
  const int i = threadIdx.x;
  const bool bad = i < n_words && image[i] != expect[i];
  if (__any(bad) && i == 0) atomicOr(flag, bit);
}

}  // namespace

hipError_t launch_fill_words(uint32_t* p, size_t n, uint32_t value, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const size_t blocks = std::min<size_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(fill_words, dim3((unsigned)blocks), dim3(256), 0, s, p, n, value);
  return hipGetLastError();
}

hipError_t launch_check_guards(const char* base, const uint64_t* offs, int n_guards, int words,
                               uint32_t value, int* flag, int bit, hipStream_t s) {
  if (n_guards <= 0) return hipSuccess;
  hipLaunchKernelGGL(check_guards, dim3(n_guards), dim3(64), 0, s, base, offs, words, value, flag, bit);
  return hipGetLastError();
}

hipError_t launch_bf16_to_f16(const void* src, void* dst, size_t n, hipStream_t s) {
  if (n % 2) return hipErrorInvalidValue;
  if (n == 0) return hipSuccess;
  const size_t blocks = std::min<size_t>((n / 2 + 255) / 256, 8192);
  hipLaunchKernelGGL(bf16_to_f16, dim3((unsigned)blocks), dim3(256), 0, s, (const uint32_t*)src,
                     (uint32_t*)dst, n / 2);
  return hipGetLastError();
}

hipError_t launch_check_header(const uint32_t* image, const uint32_t* expect, int n_words, int* flag,
                               int bit, hipStream_t s) {
  if (n_words > 64) return hipErrorInvalidValue;
  hipLaunchKernelGGL(check_header, dim3(1), dim3(64), 0, s, image, expect, n_words, flag, bit);
  return hipGetLastError();
}

hipError_t launch_rmsnorm_rows(DType in_dt, DType gain_dt, DType out_dt, const void* x,
                               int64_t ld_x, const void* gain, const void* gain2, void* out,
                               int64_t ld_out, int rows, int d, float eps, int* status,
                               hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (d % 4 || d > 1024 * kRowChunks || ld_x % 4 || ld_out % 4) return hipErrorInvalidValue;
  const dim3 grid(rows), block(256);
  auto run = [&](auto ch) {
    constexpr int CH = decltype(ch)::value;
    if (in_dt == kBF16 && gain_dt == kBF16 && out_dt == kF16)
      hipLaunchKernelGGL((rmsnorm_rows<bf16, bf16, f16, CH>), grid, block, 0, s, (const bf16*)x, ld_x,
                         (const bf16*)gain, (const bf16*)gain2, (f16*)out, ld_out, d, eps, status);
    else if (in_dt == kF32 && gain_dt == kBF16 && out_dt == kF16)
      hipLaunchKernelGGL((rmsnorm_rows<float, bf16, f16, CH>), grid, block, 0, s, (const float*)x, ld_x,
                         (const bf16*)gain, (const bf16*)gain2, (f16*)out, ld_out, d, eps, status);
    else if (in_dt == kF32 && gain_dt == kF32 && out_dt == kF32)
      hipLaunchKernelGGL((rmsnorm_rows<float, float, float, CH>), grid, block, 0, s, (const float*)x, ld_x,
                         (const float*)gain, (const float*)gain2, (float*)out, ld_out, d, eps, status);
    else
      return hipErrorInvalidValue;
    return hipGetLastError();
  };
  const int ch = (d + 1023) / 1024;
  if (ch <= 1) return run(std::integral_constant<int, 1>{});
  if (ch <= 2) return run(std::integral_constant<int, 2>{});
  if (ch <= 3) return run(std::integral_constant<int, 3>{});
  if (ch <= 4) return run(std::integral_constant<int, 4>{});
  if (ch <= 5) return run(std::integral_constant<int, 5>{});
  if (ch <= 8) return run(std::integral_constant<int, 8>{});
  return run(std::integral_constant<int, kRowChunks>{});
}

hipError_t launch_rope_scatter(DType dt, const RopeParams& p, int batch, hipStream_t s) {
  if (p.hd > 128 || p.hd % 4 || p.k < 1) return hipErrorInvalidValue;
  // rows per workgroup: doubled while the grid keeps two workgroups per compute unit
  const int cus = p.num_cus > 0 ? p.num_cus : 256;
  int rpb = 1;
  while (2 * rpb <= kRopeRows && 2 * rpb <= p.k && (int64_t)((p.k + 2 * rpb - 1) / (2 * rpb)) * batch >= 2 * cus)
    rpb *= 2;
  const dim3 grid((p.k + rpb - 1) / rpb, batch), block(256);
  if (dt == kBF16)
    hipLaunchKernelGGL((rope_scatter<bf16, true>), grid, block, 0, s, p, rpb);
  else if (dt == kF32)
    hipLaunchKernelGGL((rope_scatter<float, false>), grid, block, 0, s, p, rpb);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_scale_rows_f16(const void* x, int64_t ld_x, void* out, float* inv_scale, int rows,
                                 int cols, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(scale_rows_f16, dim3(rows), dim3(256), 0, s, (const bf16*)x, ld_x, (f16*)out,
                     inv_scale, cols);
  return hipGetLastError();
}

hipError_t launch_final_classifier(DType dt, const ClsParams& p, int batch, hipStream_t s) {
  if (p.d % 4 || p.d > 1024 * kRowChunks) return hipErrorInvalidValue;
  const dim3 grid(batch, p.n_tasks * p.n_classes);
  if (dt == kBF16)
    hipLaunchKernelGGL(final_classifier<bf16>, grid, dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL(final_classifier<float>, grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_validate(const ValidateParams& p, int batch, hipStream_t s) {
  hipLaunchKernelGGL(validate_meta, dim3(batch), dim3(64), 0, s, p);
  return hipGetLastError();
}

}  // namespace sp
