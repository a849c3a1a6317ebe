// Row kernels of the probe forward: RMSNorm, RoPE at positions N_b + j with the
// scatter into the attention layouts, final norm + read-out + linear
// classifier, and the debug validation of device-resident metadata.
#include "common.h"
#include "kernels.h"

namespace sp {
namespace {

// ---------------------------------------------------------------- RMSNorm
template <typename TI, typename TG, typename TO>
__global__ __launch_bounds__(256) void rmsnorm_rows(const TI* x, const TG* gain, TO* out, int d,
                                                    float eps) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  const TI* xr = x + (int64_t)r * d;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) {
    const float v = to_f32(xr[i]);
    ss += v * v;
  }
  ss = block_sum_256(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  TO* orow = out + (int64_t)r * d;
  for (int i = threadIdx.x; i < d; i += 256) orow[i] = from_f32<TO>(to_f32(xr[i]) * inv * to_f32(gain[i]));
}

// ---------------------------------------------------------------- RoPE + scatter
// grid (k, n_q + 2 n_kv, B), hd/2 threads: thread i rotates the pair (i, i + hd/2)
// of head h of soft row j by (N_b + j) * base^(-2i/hd), the angle in fp64.
// SPLIT (T = bf16): each value x is stored as hi = bf16(x) and lo = bf16(x - hi).
template <typename T, bool SPLIT>
__device__ __forceinline__ void put(void* hi, void* lo, int64_t idx, float x) {
  const T h = from_f32<T>(x);
  ((T*)hi)[idx] = h;
  if (SPLIT) ((T*)lo)[idx] = from_f32<T>(x - to_f32(h));
}

template <typename T, bool SPLIT>
__global__ void rope_scatter(const RopeParams p) {
  const int j = blockIdx.x, h = blockIdx.y, b = blockIdx.z, i = threadIdx.x;
  if (p.err && *p.err) return;
  const int hd = p.hd, half = hd / 2;
  const float* row = p.qkv + (int64_t)j * (p.n_q + 2 * p.n_kv) * hd;
  if (h >= p.n_q + p.n_kv) {  // value head: no rotation, the same for every sequence
    if (b != 0) return;
    const int g = h - p.n_q - p.n_kv;
    const int64_t base = (int64_t)g * hd * p.ks;
    put<T, SPLIT>(p.v_soft, p.v_soft_lo, base + (int64_t)i * p.ks + j, row[h * hd + i]);
    put<T, SPLIT>(p.v_soft, p.v_soft_lo, base + (int64_t)(i + half) * p.ks + j, row[h * hd + i + half]);
    return;
  }
  int n = p.seq_lens[b];
  n = n < 0 ? 0 : (n > p.max_seq_len ? p.max_seq_len : n);
  const double theta = pow(p.rope_base, -2.0 * (double)i / (double)hd);
  const double ang = (double)(n + j) * theta;
  const float c = (float)cos(ang), s = (float)sin(ang);
  const float x0 = row[h * hd + i], x1 = row[h * hd + i + half];
  const float r0 = x0 * c - x1 * s, r1 = x1 * c + x0 * s;
  if (h < p.n_q) {
    const int g = h / p.group, rr = j * p.group + h % p.group;
    const int64_t base = (((int64_t)b * p.n_kv + g) * p.r_alloc + rr) * hd;
    put<T, SPLIT>(p.q, p.q_lo, base + i, r0 * p.q_scale);
    put<T, SPLIT>(p.q, p.q_lo, base + i + half, r1 * p.q_scale);
  } else {
    constexpr int X = 16 / sizeof(T);
    const int g = h - p.n_q;
    const int64_t base = ((int64_t)b * p.n_kv + g) * p.ks * hd;
    const int i1 = i + half;
    put<T, SPLIT>(p.k_soft, p.k_soft_lo, base + ((int64_t)(i / X) * p.ks + j) * X + i % X, r0);
    put<T, SPLIT>(p.k_soft, p.k_soft_lo, base + ((int64_t)(i1 / X) * p.ks + j) * X + i1 % X, r1);
  }
}

// ---------------------------------------------------------------- read-out
// One workgroup per sequence: f_j = RMSNorm(y_j; gamma_final) for the read-out
// rows (the last soft row, or all k for the mean), pooled in LDS, then
// logits[c] = sum_i W_cls[c][i] pooled[i] (+ b[c]).
template <typename T>
__global__ __launch_bounds__(256) void final_classifier(const ClsParams p) {
  extern __shared__ float pooled[];
  __shared__ float red[4];
  const int b = blockIdx.x, d = p.d;
  for (int i = threadIdx.x; i < d; i += 256) pooled[i] = 0.f;
  const int j0 = p.pool_mean ? 0 : p.k - 1;
  const float w = p.pool_mean ? 1.0f / (float)p.k : 1.0f;
  for (int j = j0; j < p.k; ++j) {
    const float* yr = p.y + ((int64_t)b * p.k + j) * d;
    float ss = 0.f;
    for (int i = threadIdx.x; i < d; i += 256) ss += yr[i] * yr[i];
    ss = block_sum_256(ss, red);
    const float inv = 1.0f / sqrtf(ss / (float)d + p.eps);
    for (int i = threadIdx.x; i < d; i += 256)
      pooled[i] += yr[i] * inv * to_f32(((const T*)p.final_norm)[i]) * w;
  }
  __syncthreads();
  for (int c = 0; c < p.n_classes; ++c) {
    const T* wr = (const T*)p.w_cls + (int64_t)c * d;
    float acc = 0.f;
    for (int i = threadIdx.x; i < d; i += 256) acc += to_f32(wr[i]) * pooled[i];
    acc = block_sum_256(acc, red);
    if (threadIdx.x == 0) p.logits[(int64_t)b * p.n_classes + c] = acc + (p.b_cls ? p.b_cls[c] : 0.f);
  }
}

// ---------------------------------------------------------------- validation
__global__ void validate_meta(const ValidateParams p) {
  const int b = blockIdx.x;
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

}  // namespace

hipError_t launch_rmsnorm_rows(DType in_dt, DType gain_dt, DType out_dt, const void* x,
                               const void* gain, void* out, int rows, int d, float eps,
                               hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const dim3 grid(rows), block(256);
  if (in_dt == kBF16 && gain_dt == kBF16 && out_dt == kF16)
    hipLaunchKernelGGL((rmsnorm_rows<bf16, bf16, f16>), grid, block, 0, s, (const bf16*)x, (const bf16*)gain, (f16*)out, d, eps);
  else if (in_dt == kF32 && gain_dt == kBF16 && out_dt == kF16)
    hipLaunchKernelGGL((rmsnorm_rows<float, bf16, f16>), grid, block, 0, s, (const float*)x, (const bf16*)gain, (f16*)out, d, eps);
  else if (in_dt == kF32 && gain_dt == kF32 && out_dt == kF32)
    hipLaunchKernelGGL((rmsnorm_rows<float, float, float>), grid, block, 0, s, (const float*)x, (const float*)gain, (float*)out, d, eps);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_rope_scatter(DType dt, const RopeParams& p, int batch, hipStream_t s) {
  const dim3 grid(p.k, p.n_q + 2 * p.n_kv, batch), block(p.hd / 2);
  if (dt == kBF16)
    hipLaunchKernelGGL((rope_scatter<bf16, true>), grid, block, 0, s, p);
  else if (dt == kF32)
    hipLaunchKernelGGL((rope_scatter<float, false>), grid, block, 0, s, p);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_final_classifier(DType dt, const ClsParams& p, int batch, hipStream_t s) {
  const size_t lds = (size_t)p.d * sizeof(float);
  if (dt == kBF16)
    hipLaunchKernelGGL(final_classifier<bf16>, dim3(batch), dim3(256), lds, s, p);
  else
    hipLaunchKernelGGL(final_classifier<float>, dim3(batch), dim3(256), lds, s, p);
  return hipGetLastError();
}

hipError_t launch_validate(const ValidateParams& p, int batch, hipStream_t s) {
  hipLaunchKernelGGL(validate_meta, dim3(batch), dim3(64), 0, s, p);
  return hipGetLastError();
}

}  // namespace sp
