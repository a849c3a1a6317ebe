// Projections of the probe's decoder layer: C = A W^T with A [M][K] and the
// weight W [N][K] both K-contiguous, fused epilogues (residual adds, SwiGLU).
//
// bf16 path: fp16 activations A, bf16 weights converted exactly to fp16 while
// they are staged into LDS (|w| in [2^-14, 65504]), v_mfma_f32_16x16x32_f16 with
// fp32 accumulation.  256 threads as 2 x 2 waves, a BM x BN x 64 tile staged in
// LDS (rows padded by 16 bytes so the 16 lanes of an MFMA fragment read hit
// distinct banks), two LDS buffers: the next K-step is fetched into registers
// while the current one runs on the matrix cores.
// SwiGLU: the BN weight rows of a tile alternate 16 gate rows and the 16
// matching up rows, so every lane holds gate and up of the same outputs.
#include "common.h"
#include "kernels.h"

namespace sp {
namespace {

template <int EPI>
__device__ __forceinline__ const bf16* weight_row(const GemmParams& p, int tile_n0, int rho,
                                                  int n_blk, int BN) {
  if (EPI == kEpiSwiglu) {
    const int pair = rho >> 5, w = rho & 31;
    const int out = n_blk * (BN / 2) + 16 * pair + (w & 15);
    return (const bf16*)(w < 16 ? p.b[0] : p.b[1]) + (int64_t)out * p.ldb;
  }
  const int n = tile_n0 + rho;
  if (n < p.b_split0) return (const bf16*)p.b[0] + (int64_t)n * p.ldb;
  if (n < p.b_split1) return (const bf16*)p.b[1] + (int64_t)(n - p.b_split0) * p.ldb;
  return (const bf16*)p.b[2] + (int64_t)(n - p.b_split1) * p.ldb;
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

template <int BM, int BN, int EPI>
__global__ __launch_bounds__(256) void gemm_mfma(const GemmParams p) {
  constexpr int BK = 64, LD = BK + 8;
  constexpr int WM = BM / 2, WN = BN / 2, MT = WM / 16, NT = WN / 16;
  constexpr int AU = BM * 8 / 256, BU = BN * 8 / 256;  // 16-byte chunks per thread
  static_assert(AU >= 1 && BU >= 1, "tile too small");
  __shared__ __attribute__((aligned(16))) f16 As[2][BM * LD];
  __shared__ __attribute__((aligned(16))) f16 Bs[2][BN * LD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, li = lane & 15, la = lane >> 4;
  const int n_blk = blockIdx.x, m0 = blockIdx.y * BM, n0 = n_blk * BN;
  const f16* A = (const f16*)p.a;

  const f16* arow[AU];
  const bf16* brow[BU];
  int aoff[AU], boff[BU];
#pragma unroll
  for (int u = 0; u < AU; ++u) {
    const int q = tid + 256 * u, row = q >> 3;
    const int gm = m0 + row < p.M ? m0 + row : p.M - 1;  // rows past M re-read row M-1; never stored
    arow[u] = A + (int64_t)gm * p.lda + (q & 7) * 8;
    aoff[u] = row * LD + (q & 7) * 8;
  }
#pragma unroll
  for (int u = 0; u < BU; ++u) {
    const int q = tid + 256 * u, row = q >> 3;
    brow[u] = weight_row<EPI>(p, n0, row, n_blk, BN) + (q & 7) * 8;
    boff[u] = row * LD + (q & 7) * 8;
  }

  uint4 ra[AU], rb[BU];
  auto gload = [&](int kt) {
    const int k0 = kt * BK;
#pragma unroll
    for (int u = 0; u < AU; ++u) ra[u] = ld16(arow[u] + k0);
#pragma unroll
    for (int u = 0; u < BU; ++u) rb[u] = bf16x8_to_f16x8(ld16(brow[u] + k0));
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int u = 0; u < AU; ++u) st16(&As[buf][aoff[u]], ra[u]);
#pragma unroll
    for (int u = 0; u < BU; ++u) st16(&Bs[buf][boff[u]], rb[u]);
  };

  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int KT = p.K / BK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) gload(kt + 1);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      f16x8 af[MT], bfr[NT];
#pragma unroll
      for (int i = 0; i < MT; ++i)
        af[i] = as_f16x8(ld16(&As[buf][(wm * WM + 16 * i + li) * LD + kk * 32 + 8 * la]));
#pragma unroll
      for (int j = 0; j < NT; ++j)
        bfr[j] = as_f16x8(ld16(&Bs[buf][(wn * WN + 16 * j + li) * LD + kk * 32 + 8 * la]));
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[i][j] = mfma16x16x32(af[i], bfr[j], acc[i][j]);
    }
    if (kt + 1 < KT) lstore(buf ^ 1);
    __syncthreads();
  }

  // Lane holds C[16i + 4la + r][16j + li] of the wave tile.
#pragma unroll
  for (int i = 0; i < MT; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + wm * WM + 16 * i + 4 * la + r;
      if (m >= p.M) continue;
      if (EPI == kEpiSwiglu) {
#pragma unroll
        for (int j = 0; j < NT; j += 2) {
          const int pair = (wn * WN + 16 * j) >> 5;
          const int n = n_blk * (BN / 2) + 16 * pair + li;
          const float gt = acc[i][j][r], up = acc[i][j + 1][r];
          ((f16*)p.c)[(int64_t)m * p.ldc + n] = (f16)(silu(gt) * up);
        }
      } else {
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          const int n = n0 + wn * WN + 16 * j + li;
          float v = acc[i][j][r];
          if (EPI == kEpiResidRow)
            v += (float)((const bf16*)p.r)[(int64_t)(m % p.r_mod) * p.N + n];
          else if (EPI == kEpiResidF32)
            v += ((const float*)p.r)[(int64_t)m * p.ldc + n];
          ((float*)p.c)[(int64_t)m * p.ldc + n] = v;
        }
      }
    }
  }
}

// ---------------------------------------------------------------- fp32 path
// One thread per output, the dot product in order k = 0..K-1.
template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32(const GemmParams p) {
  const int n = blockIdx.x * 256 + threadIdx.x, m = blockIdx.y;
  const int n_out = EPI == kEpiSwiglu ? p.N / 2 : p.N;
  if (n >= n_out) return;
  const float* a = (const float*)p.a + (int64_t)m * p.lda;
  auto row = [&](int nn) -> const float* {
    if (nn < p.b_split0) return (const float*)p.b[0] + (int64_t)nn * p.ldb;
    if (nn < p.b_split1) return (const float*)p.b[1] + (int64_t)(nn - p.b_split0) * p.ldb;
    return (const float*)p.b[2] + (int64_t)(nn - p.b_split1) * p.ldb;
  };
  if (EPI == kEpiSwiglu) {
    const float* wg = (const float*)p.b[0] + (int64_t)n * p.ldb;
    const float* wu = (const float*)p.b[1] + (int64_t)n * p.ldb;
    float g = 0.f, u = 0.f;
    for (int k = 0; k < p.K; ++k) {
      g += a[k] * wg[k];
      u += a[k] * wu[k];
    }
    ((float*)p.c)[(int64_t)m * p.ldc + n] = g / (1.0f + expf(-g)) * u;
    return;
  }
  const float* w = row(n);
  float acc = 0.f;
  for (int k = 0; k < p.K; ++k) acc += a[k] * w[k];
  if (EPI == kEpiResidRow) acc += ((const float*)p.r)[(int64_t)(m % p.r_mod) * p.N + n];
  if (EPI == kEpiResidF32) acc += ((const float*)p.r)[(int64_t)m * p.ldc + n];
  ((float*)p.c)[(int64_t)m * p.ldc + n] = acc;
}

template <int BM, int BN>
hipError_t launch_mfma_tile(Epilogue epi, const GemmParams& p, hipStream_t s) {
  const dim3 grid(p.N / BN, (p.M + BM - 1) / BM);
  switch (epi) {
    case kEpiStore: hipLaunchKernelGGL((gemm_mfma<BM, BN, kEpiStore>), grid, dim3(256), 0, s, p); break;
    case kEpiResidRow: hipLaunchKernelGGL((gemm_mfma<BM, BN, kEpiResidRow>), grid, dim3(256), 0, s, p); break;
    case kEpiResidF32: hipLaunchKernelGGL((gemm_mfma<BM, BN, kEpiResidF32>), grid, dim3(256), 0, s, p); break;
    case kEpiSwiglu: hipLaunchKernelGGL((gemm_mfma<BM, BN, kEpiSwiglu>), grid, dim3(256), 0, s, p); break;
  }
  return hipGetLastError();
}

bool tile_ok(const GemmParams& p, Epilogue epi, int BN) {
  if (p.N % BN) return false;
  if (epi == kEpiSwiglu) return BN >= 64;
  return p.b_split0 % BN == 0 && p.b_split1 % BN == 0;
}

}  // namespace

hipError_t launch_gemm(DType dt, Epilogue epi, const GemmParams& p, hipStream_t s) {
  if (p.M <= 0) return hipSuccess;
  if (dt == kF32) {
    const int n_out = epi == kEpiSwiglu ? p.N / 2 : p.N;
    const dim3 grid((n_out + 255) / 256, p.M);
    switch (epi) {
      case kEpiStore: hipLaunchKernelGGL(gemm_f32<kEpiStore>, grid, dim3(256), 0, s, p); break;
      case kEpiResidRow: hipLaunchKernelGGL(gemm_f32<kEpiResidRow>, grid, dim3(256), 0, s, p); break;
      case kEpiResidF32: hipLaunchKernelGGL(gemm_f32<kEpiResidF32>, grid, dim3(256), 0, s, p); break;
      case kEpiSwiglu: hipLaunchKernelGGL(gemm_f32<kEpiSwiglu>, grid, dim3(256), 0, s, p); break;
    }
    return hipGetLastError();
  }
  if (p.K % 64) return hipErrorInvalidValue;
  // Largest tile that still gives one workgroup per compute unit (256), else the
  // tile with the most workgroups.
  struct Cand { int bm, bn; };
  const Cand cands[4] = {{128, 128}, {64, 128}, {32, 128}, {32, 64}};
  int best = -1;
  long best_tiles = -1;
  for (int c = 0; c < 4; ++c) {
    if (!tile_ok(p, epi, cands[c].bn)) continue;
    const long tiles = (long)((p.M + cands[c].bm - 1) / cands[c].bm) * (p.N / cands[c].bn);
    if (tiles >= 256) { best = c; break; }
    if (tiles > best_tiles) { best_tiles = tiles; best = c; }
  }
  switch (best) {
    case 0: return launch_mfma_tile<128, 128>(epi, p, s);
    case 1: return launch_mfma_tile<64, 128>(epi, p, s);
    case 2: return launch_mfma_tile<32, 128>(epi, p, s);
    case 3: return launch_mfma_tile<32, 64>(epi, p, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace sp
