// Projections of the probe's decoder layer: C = A W^T with A [M][K] and the
// weight W [N][K] both K-contiguous, fused epilogues (residual adds, SwiGLU).
//
// bf16 path: fp16 activations A, bf16 weights, v_mfma_f32_16x16x32_f16 with
// fp32 accumulation.  A workgroup computes a BM x BN tile with WGM x WGN waves
// (each a (BM/WGM) x (BN/WGN) sub-tile) and consumes K in steps of BK (32 or
// 64: one or two MFMAs deep).  Each step's A and W tiles are loaded straight
// into LDS, S - 1 steps ahead of use, through an S-stage ring (one barrier per
// step; S = 2 is plain double buffering: the loads of step k + 1 are issued
// right after the barrier of step k and waited for before the next); weights stay bf16 in LDS and are converted exactly to fp16 (|w| in
// [2^-14, 65504]) as a wave reads its fragments.  A row of a stage tile is BK
// values = PPR 16-byte pieces; piece kp of row r sits at
//   r * PPR + (kp ^ ((r >> 1) & (PPR - 1)))
// which leaves the 16-byte fragment reads of 16 consecutive rows free of LDS
// bank conflicts for both PPR = 4 and 8 (the LDS bank-conflict counter reads 0;
// a shift of 2 for PPR = 4 measured conflicts on half the LDS cycles).
// SwiGLU: the BN weight rows of a tile alternate 16 gate rows and the 16
// matching up rows, so every lane holds gate and up of the same outputs.
// Split-K (PART, small M: the product then streams the weights with too few
// workgroups to keep enough loads in flight): blockIdx.y takes a slice of the
// K steps and writes its fp32 partial tile; gemm_reduce sums the slices in a
// fixed order and applies the epilogue.
// Weights come either as the caller's bf16 matrices (WBF16, converted per
// fragment) or as an fp16 image of them made once for the frozen head (no
// conversion: the same values, so the same results bit for bit).
// Tile order: workgroups are dealt to the XCDs round-robin (launch index mod
// the XCD count).  The launch index is re-mapped so that each XCD takes a
// contiguous run of a grouped tile order (group_m row tiles, then the next
// column tile): the workgroups that share an XCD's L2 at one time then cover a
// compact block of group_m row tiles by (CUs per XCD / group_m) column tiles,
// instead of every row tile of one column tile, and fetch far fewer operand
// bytes from beyond the L2 (27B-shaped gate/up on 8192 rows: 15% faster).
#include "common.h"
#include "kernels.h"

namespace sp {
namespace {

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

// Tile (m_tile, n_tile) of launch index L among nwg tiles (see the tile order above).
__device__ __forceinline__ void tile_of(int L, int nwg, int mtiles, int ntiles, int n_xcd, int group_m,
                                        int& m_tile, int& n_tile) {
  const int x = L % n_xcd, r = L / n_xcd;
  const int q = nwg / n_xcd, rem = nwg % n_xcd;
  const int t = (x < rem ? x * (q + 1) : rem * (q + 1) + (x - rem) * q) + r;
  const int per_group = group_m * ntiles;
  const int g = t / per_group, in = t - g * per_group;
  const int gm = min(group_m, mtiles - g * group_m);  // the last group may hold fewer row tiles
  m_tile = g * group_m + in % gm;
  n_tile = in / gm;
}

template <int BM, int BN, int WGM, int WGN, int S, int BK, int EPI, bool PART, bool WBF16>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_lds(const GemmParams p) {
  constexpr int NW = WGM * WGN, WM = BM / WGM, WN = BN / WGN, MT = WM / 16, NT = WN / 16;
  constexpr int PPR = BK / 8;                        // 16-byte pieces per tile row
  constexpr int RPI = 64 / PPR;                      // tile rows per 64-piece load
  constexpr int SWS = 1;                             // swizzle: kp ^ ((r >> SWS) & (PPR - 1))
  constexpr int NIA = BM / RPI, NI = NIA + BN / RPI;  // 64-piece loads per step
  constexpr int IPW = (NI + NW - 1) / NW;            // loads per wave per step
  constexpr int STAGE = (BM + BN) * PPR;             // pieces per stage
  static_assert(BK == 32 || BK == 64, "step depth");
  static_assert(WM % 16 == 0 && WN % 16 == 0, "wave tile");
  static_assert(S >= 2 && (S - 2) * IPW < 64, "stages");
  static_assert(EPI != kEpiSwiglu || WN % 32 == 0, "SwiGLU pairs 16 gate and 16 up columns");
  __shared__ u32x4 lds[S * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, li = lane & 15, la = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  __builtin_assume(wave >= 0 && wave < NW);
  const int wm = wave / WGN, wn = wave % WGN;

  const int mtiles = (p.M + BM - 1) / BM, ntiles = p.N / BN;
  int m_tile, n_tile;
  tile_of(blockIdx.x, gridDim.x, mtiles, ntiles, p.n_xcd, p.group_m, m_tile, n_tile);
  const int m0 = m_tile * BM, n0 = n_tile * BN;

  // This wave's loads: slots j*NW + wave (mod NI; a wave count that does not
  // divide NI re-issues a few slots with the same bytes).  Per slot: the
  // RPI-row block's base pointer (uniform), its place in the stage and the
  // lane's byte offset (fixed; each K step adds 2 BK bytes to the base).
  const char* gbase[IPW];
  int lds_piece[IPW];
  uint32_t lane_off[IPW];
  const int row_in = lane / PPR, kslot = lane % PPR;
#pragma unroll
  for (int j = 0; j < IPW; ++j) {
    const int sl = (j * NW + wave) % NI;
    const int blk = sl < NIA ? sl : sl - NIA;            // RPI-row block of the A or W tile
    const int kp = kslot ^ (((blk * RPI + row_in) >> SWS) & (PPR - 1));
    if (sl < NIA) {
      const int g = min(m0 + blk * RPI + row_in, p.M - 1);  // rows past M re-read row M-1; never stored
      gbase[j] = (const char*)p.a;
      lane_off[j] = (uint32_t)(g * p.lda * 2 + kp * 16);
      lds_piece[j] = blk * 64;
    } else {
      int src, row;
      if (EPI == kEpiSwiglu) {  // an RPI-row block lies inside one 16-row gate or up group
        const int r = blk * RPI;
        src = (r >> 4) & 1;
        row = n_tile * (BN / 2) + 16 * (r >> 5) + (r & 15) + row_in;
      } else {
        const int n = n0 + blk * RPI;  // b_split0/1 are multiples of BN
        src = n < p.b_split0 ? 0 : (n < p.b_split1 ? 1 : 2);
        row = n - (src == 0 ? 0 : (src == 1 ? p.b_split0 : p.b_split1)) + row_in;
      }
      gbase[j] = (const char*)(src == 0 ? p.b[0] : (src == 1 ? p.b[1] : p.b[2]));
      lane_off[j] = (uint32_t)(row * p.ldb * 2 + kp * 16);
      lds_piece[j] = BM * PPR + blk * 64;
    }
  }
  auto issue = [&](int kt, int stg) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < IPW; ++j)
      ld16_to_lds<false>(gbase[j] + kt * 2 * BK, lane_off[j], &lds[stg * STAGE + lds_piece[j]]);
  };

  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Steps past the last re-load the last one (into a stage no later step
  // reads), so every step issues the same loads and one vmcnt value fits all.
  const int KT = p.K / BK;
  const int kb = (int)(((int64_t)KT * blockIdx.y) / gridDim.y);       // this slice's K steps
  const int ke = (int)(((int64_t)KT * (blockIdx.y + 1)) / gridDim.y);
#pragma unroll
  for (int st = 0; st < S - 1; ++st) issue(min(kb + st, ke - 1), st);
  int stg = 0;
  for (int kt = kb; kt < ke; ++kt) {
    wait_vmcnt<(S - 2) * IPW>();  // this wave's loads of step kt have landed
    lds_barrier();                // everyone's have; everyone is done with step kt - 1
    issue(min(kt + S - 1, ke - 1), stg == 0 ? S - 1 : stg - 1);
    const u32x4* As = lds + stg * STAGE;
    const u32x4* Bs = As + BM * PPR;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      // piece 4 ks + la of rows 16x + li (the row's swizzle depends on li only)
      const int pc = (4 * ks + la) ^ ((li >> SWS) & (PPR - 1));
      f16x8 af[MT], bfr[NT];
#pragma unroll
      for (int i = 0; i < MT; ++i) af[i] = __builtin_bit_cast(f16x8, As[(wm * WM + 16 * i + li) * PPR + pc]);
#pragma unroll
      for (int j = 0; j < NT; ++j)
        bfr[j] = __builtin_bit_cast(f16x8, WBF16 ? bf16x8_to_f16x8(Bs[(wn * WN + 16 * j + li) * PPR + pc])
                                                 : Bs[(wn * WN + 16 * j + li) * PPR + pc]);
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[i][j] = mfma16x16x32(af[i], bfr[j], acc[i][j]);
    }
    if constexpr (BK == 64 && !WBF16) {
      // Instruction order of the step: the first half-step's fragment reads,
      // then the second half-step's reads one by one between the first
      // half-step's products, then the remaining products.  Left to itself the
      // compiler issued the second reads only after every product of the first
      // half, so each step waited out an LDS round trip with the matrix cores
      // idle (27B-shaped gate/up 2.30 -> 2.23 ms, o and down 2-3% faster).
      constexpr int NF = MT + NT, NM = MT * NT;
      __builtin_amdgcn_sched_group_barrier(0x100, NF, 0);  // 0x100: LDS reads
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // 0x008: MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2 * NM - NF, 0);
    }
    stg = stg == S - 1 ? 0 : stg + 1;
  }
  wait_vmcnt<0>();

  // Lane holds C[16i + 4la + r][16j + li] of the wave tile.
  bool oor = false;  // an fp16 SwiGLU output out of fp16's range
#pragma unroll
  for (int i = 0; i < MT; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + wm * WM + 16 * i + 4 * la + r;
      if (m >= p.M) continue;
      if (PART) {
        float* prow = p.part + ((int64_t)blockIdx.y * p.M + m) * p.N + n0 + wn * WN + li;
#pragma unroll
        for (int j = 0; j < NT; ++j) prow[16 * j] = acc[i][j][r];
      } else if (EPI == kEpiSwiglu) {
#pragma unroll
        for (int j = 0; j < NT; j += 2) {
          const int pair = (wn * WN + 16 * j) >> 5;
          const int n = n_tile * (BN / 2) + 16 * pair + li;
          const float gt = acc[i][j][r], up = acc[i][j + 1][r];
          const float v = silu(gt) * up;
          oor |= !(fabsf(v) <= 65504.0f);
          ((f16*)p.c)[(int64_t)m * p.ldc + n] = (f16)v;
        }
      } else {
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          const int n = n0 + wn * WN + 16 * j + li;
          float v = acc[i][j][r];
          if (EPI == kEpiResidRow)
            v += (float)((const bf16*)p.r)[(int64_t)(m % p.r_mod) * p.r_ld + n];
          else if (EPI == kEpiResidF32)
            v += ((const float*)p.r)[(int64_t)m * p.r_ld + n];
          else if (EPI == kEpiRowScale)
            v *= ((const float*)p.r)[m];
          ((float*)p.c)[(int64_t)m * p.ldc + n] = v;
        }
      }
    }
  }
  if (EPI == kEpiSwiglu && !PART && __any(oor) && lane == 0 && p.status) atomicOr(p.status, kStatusRange);
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
  if (EPI == kEpiResidRow) acc += ((const float*)p.r)[(int64_t)(m % p.r_mod) * p.r_ld + n];
  if (EPI == kEpiResidF32) acc += ((const float*)p.r)[(int64_t)m * p.r_ld + n];
  if (EPI == kEpiRowScale) acc *= ((const float*)p.r)[m];
  ((float*)p.c)[(int64_t)m * p.ldc + n] = acc;
}

// Sum of the split-K slices and the epilogue, one thread per output.  SwiGLU:
// output o of tile o / (bn/2) has its gate column 32 ((o % (bn/2)) / 16) +
// o % 16 in the tile's interleaved columns and its up column 16 later.
template <int EPI>
__global__ __launch_bounds__(256) void gemm_reduce(const GemmParams p, int ksplit, int bn) {
  const int n_out = EPI == kEpiSwiglu ? p.N / 2 : p.N;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)p.M * n_out) return;
  const int m = (int)(idx / n_out), o = (int)(idx % n_out);
  const int64_t slice = (int64_t)p.M * p.N;
  const float* src = p.part + (int64_t)m * p.N;
  if (EPI == kEpiSwiglu) {
    const int w = o % (bn / 2);
    const int g = (o / (bn / 2)) * bn + 32 * (w / 16) + w % 16;
    float gt = 0.f, up = 0.f;
    for (int k = 0; k < ksplit; ++k) {
      gt += src[k * slice + g];
      up += src[k * slice + g + 16];
    }
    const float v = silu(gt) * up;
    ((f16*)p.c)[(int64_t)m * p.ldc + o] = (f16)v;
    if (!(fabsf(v) <= 65504.0f) && p.status) atomicOr(p.status, kStatusRange);
    return;
  }
  float v = 0.f;
  for (int k = 0; k < ksplit; ++k) v += src[k * slice + o];
  if (EPI == kEpiResidRow) v += (float)((const bf16*)p.r)[(int64_t)(m % p.r_mod) * p.r_ld + o];
  if (EPI == kEpiResidF32) v += ((const float*)p.r)[(int64_t)m * p.r_ld + o];
  if (EPI == kEpiRowScale) v *= ((const float*)p.r)[m];
  ((float*)p.c)[(int64_t)m * p.ldc + o] = v;
}

// The same, four consecutive outputs per thread (16-byte partial loads) and
// one output row per blockIdx.y; the launcher takes it when every row stride
// and base keeps those accesses aligned.  Same sums in the same order.
template <int EPI>
__global__ __launch_bounds__(256) void gemm_reduce4(const GemmParams p, int ksplit, int bn) {
  const int n_out = EPI == kEpiSwiglu ? p.N / 2 : p.N;
  const int m = blockIdx.y, o = 4 * (blockIdx.x * 256 + threadIdx.x);
  if (o >= n_out) return;
  const int64_t slice = (int64_t)p.M * p.N;
  const float* src = p.part + (int64_t)m * p.N;
  if (EPI == kEpiSwiglu) {
    const int w = o % (bn / 2);  // o % 4 == 0: the four outputs share one 16-column group
    const int g = (o / (bn / 2)) * bn + 32 * (w / 16) + w % 16;
    float4 gt = make_float4(0.f, 0.f, 0.f, 0.f), up = gt;
    for (int k = 0; k < ksplit; ++k) {
      const float4 a = *reinterpret_cast<const float4*>(src + k * slice + g);
      const float4 u = *reinterpret_cast<const float4*>(src + k * slice + g + 16);
      gt.x += a.x; gt.y += a.y; gt.z += a.z; gt.w += a.w;
      up.x += u.x; up.y += u.y; up.z += u.z; up.w += u.w;
    }
    const float v[4] = {silu(gt.x) * up.x, silu(gt.y) * up.y, silu(gt.z) * up.z, silu(gt.w) * up.w};
    f16x4 h;
    bool oor = false;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      h[e] = (f16)v[e];
      oor |= !(fabsf(v[e]) <= 65504.0f);
    }
    *reinterpret_cast<f16x4*>((f16*)p.c + (int64_t)m * p.ldc + o) = h;
    if (oor && p.status) atomicOr(p.status, kStatusRange);
    return;
  }
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int k = 0; k < ksplit; ++k) {
    const float4 a = *reinterpret_cast<const float4*>(src + k * slice + o);
    v.x += a.x; v.y += a.y; v.z += a.z; v.w += a.w;
  }
  if (EPI == kEpiResidRow) {
    const bf16* rr = (const bf16*)p.r + (int64_t)(m % p.r_mod) * p.r_ld + o;
    v.x += (float)rr[0]; v.y += (float)rr[1]; v.z += (float)rr[2]; v.w += (float)rr[3];
  }
  if (EPI == kEpiResidF32) {
    const float4 r = *reinterpret_cast<const float4*>((const float*)p.r + (int64_t)m * p.r_ld + o);
    v.x += r.x; v.y += r.y; v.z += r.z; v.w += r.w;
  }
  if (EPI == kEpiRowScale) {
    const float sc = ((const float*)p.r)[m];
    v.x *= sc; v.y *= sc; v.z *= sc; v.w *= sc;
  }
  *reinterpret_cast<float4*>((float*)p.c + (int64_t)m * p.ldc + o) = v;
}

template <int BM, int BN, int WGM, int WGN, int S, int BK, bool PART, bool WB>
hipError_t launch_tile_k(Epilogue epi, const GemmParams& p, dim3 grid, hipStream_t s) {
  const dim3 block(64 * WGM * WGN);
  switch (epi) {
    case kEpiStore: hipLaunchKernelGGL((gemm_lds<BM, BN, WGM, WGN, S, BK, kEpiStore, PART, WB>), grid, block, 0, s, p); break;
    case kEpiResidRow: hipLaunchKernelGGL((gemm_lds<BM, BN, WGM, WGN, S, BK, kEpiResidRow, PART, WB>), grid, block, 0, s, p); break;
    case kEpiResidF32: hipLaunchKernelGGL((gemm_lds<BM, BN, WGM, WGN, S, BK, kEpiResidF32, PART, WB>), grid, block, 0, s, p); break;
    case kEpiRowScale: hipLaunchKernelGGL((gemm_lds<BM, BN, WGM, WGN, S, BK, kEpiRowScale, PART, WB>), grid, block, 0, s, p); break;
    case kEpiSwiglu:
      if constexpr ((BN / WGN) % 32 == 0)
        hipLaunchKernelGGL((gemm_lds<BM, BN, WGM, WGN, S, BK, kEpiSwiglu, PART, WB>), grid, block, 0, s, p);
      else
        return hipErrorInvalidValue;
      break;
  }
  return hipGetLastError();
}

// K split ksplit ways (ksplit > 1: fp32 partials in p.part, then gemm_reduce).
template <int BM, int BN, int WGM, int WGN, int S, int BK>
hipError_t launch_tile(Epilogue epi, const GemmParams& p, int ksplit, hipStream_t s) {
  if (p.K % BK || p.K / BK < ksplit) return hipErrorInvalidValue;  // slices of whole steps, maybe uneven
  const dim3 grid(((p.M + BM - 1) / BM) * (p.N / BN), ksplit);
  hipError_t e;
  if (ksplit > 1)
    e = p.b_f16 ? launch_tile_k<BM, BN, WGM, WGN, S, BK, true, false>(epi, p, grid, s)
                : launch_tile_k<BM, BN, WGM, WGN, S, BK, true, true>(epi, p, grid, s);
  else
    e = p.b_f16 ? launch_tile_k<BM, BN, WGM, WGN, S, BK, false, false>(epi, p, grid, s)
                : launch_tile_k<BM, BN, WGM, WGN, S, BK, false, true>(epi, p, grid, s);
  if (e != hipSuccess || ksplit == 1) return e;
  return launch_gemm_reduce(epi, p, ksplit, BN, s);
}

// Tile shapes (BM, BN, waves along M, waves along N, K-step depth); the stage
// counts are in launch_tile_index.  The residual epilogues (o, down) prefer
// 256 x 128 tiles with 64-deep steps, which at 2048-8192 rows take half the
// time of 128 x 64.  Index 9 is the 32 x 128 tile of the 17-32-row products.
// Index 10 is 256 x 256 with 64-deep steps, double-buffered (two 64 KB stages):
// 64-deep steps halve the barriers per unit of K and load whole 128-byte rows
// per step (32-deep steps load half rows, and with them half cache lines), and
// more stages measured no faster (SwiGLU, fp16 weights, 8192 x 34816 x 5120:
// 2.35 ms against 2.59 ms for 256 x 256 in 32-deep steps; 2048 x 24576 x 4096:
// 0.335 ms against 0.368 ms).  Index 11 is 256 x 160 in three 52 KB stages, for
// residual products whose 256 x 256 or 256 x 128 grids end in a partial round
// (8192 x 5120: 1024 tiles, four whole rounds); index 12 is 256 x 192 with
// 64-deep steps, double-buffered, for SwiGLU grids of one round (512 x 24576 x
// 4096: 119 us against 124 us in 32-deep steps).
struct TileShape { int bm, bn, wgm, wgn, bk; };
constexpr int kNumTiles = 13;
constexpr TileShape kTiles[kNumTiles] = {
    {256, 256, 2, 4, 32}, {256, 192, 4, 2, 32}, {256, 128, 4, 2, 64}, {128, 64, 4, 2, 64},
    {64, 64, 2, 2, 64},   {32, 64, 1, 2, 64},   {16, 32, 1, 1, 64},  {16, 16, 1, 1, 64},
    {16, 32, 1, 1, 32},   {32, 128, 1, 4, 64},  {256, 256, 4, 2, 64}, {256, 160, 4, 2, 64},
    {256, 192, 4, 2, 64}};
constexpr int kOrderSwiglu[9] = {0, 1, 2, 3, 4, 5, 6, 7, 8};
constexpr int kOrderResid[9] = {2, 1, 0, 3, 4, 5, 6, 7, 8};

bool tile_ok(const GemmParams& p, Epilogue epi, const TileShape& t) {
  if (p.N % t.bn || p.K % t.bk) return false;
  if (epi == kEpiSwiglu) return (t.bn / t.wgn) % 32 == 0;
  return p.b_split0 % t.bn == 0 && p.b_split1 % t.bn == 0;
}

hipError_t launch_tile_index(int c, Epilogue epi, const GemmParams& p, int ksplit, hipStream_t s) {
  switch (c) {
    case 0: return launch_tile<256, 256, 2, 4, 3, 32>(epi, p, ksplit, s);
    case 1: return launch_tile<256, 192, 4, 2, 3, 32>(epi, p, ksplit, s);
    case 2: return launch_tile<256, 128, 4, 2, 3, 64>(epi, p, ksplit, s);
    case 3: return launch_tile<128, 64, 4, 2, 6, 64>(epi, p, ksplit, s);
    case 4: return launch_tile<64, 64, 2, 2, 8, 64>(epi, p, ksplit, s);
    case 5: return launch_tile<32, 64, 1, 2, 8, 64>(epi, p, ksplit, s);
    case 6: return launch_tile<16, 32, 1, 1, 8, 64>(epi, p, ksplit, s);
    case 7: return launch_tile<16, 16, 1, 1, 8, 64>(epi, p, ksplit, s);
    case 8: return launch_tile<16, 32, 1, 1, 8, 32>(epi, p, ksplit, s);
    case 9: return launch_tile<32, 128, 1, 4, 6, 64>(epi, p, ksplit, s);
    case 10: return launch_tile<256, 256, 4, 2, 2, 64>(epi, p, ksplit, s);
    case 11: return launch_tile<256, 160, 4, 2, 3, 64>(epi, p, ksplit, s);
    case 12: return launch_tile<256, 192, 4, 2, 2, 64>(epi, p, ksplit, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_gemm_reduce(Epilogue epi, const GemmParams& p, int ksplit, int bn, hipStream_t s) {
  const int n_out = epi == kEpiSwiglu ? p.N / 2 : p.N;
  auto al16 = [](const void* q) { return ((uintptr_t)q & 15) == 0; };
  const bool vec = n_out % 4 == 0 && p.N % 4 == 0 && p.ldc % 4 == 0 && al16(p.part) &&
                   (epi == kEpiSwiglu ? ((uintptr_t)p.c & 7) == 0 && bn % 32 == 0 : al16(p.c)) &&
                   (epi == kEpiResidRow ? p.r_ld % 4 == 0 && ((uintptr_t)p.r & 7) == 0 : true) &&
                   (epi == kEpiResidF32 ? p.r_ld % 4 == 0 && al16(p.r) : true) && p.M <= 65535;
  if (vec) {
    const dim3 g4((unsigned)((n_out / 4 + 255) / 256), (unsigned)p.M);
    switch (epi) {
      case kEpiStore: hipLaunchKernelGGL(gemm_reduce4<kEpiStore>, g4, dim3(256), 0, s, p, ksplit, bn); break;
      case kEpiResidRow: hipLaunchKernelGGL(gemm_reduce4<kEpiResidRow>, g4, dim3(256), 0, s, p, ksplit, bn); break;
      case kEpiResidF32: hipLaunchKernelGGL(gemm_reduce4<kEpiResidF32>, g4, dim3(256), 0, s, p, ksplit, bn); break;
      case kEpiRowScale: hipLaunchKernelGGL(gemm_reduce4<kEpiRowScale>, g4, dim3(256), 0, s, p, ksplit, bn); break;
      case kEpiSwiglu: hipLaunchKernelGGL(gemm_reduce4<kEpiSwiglu>, g4, dim3(256), 0, s, p, ksplit, bn); break;
    }
    return hipGetLastError();
  }
  const dim3 rgrid((unsigned)(((int64_t)p.M * n_out + 255) / 256));
  switch (epi) {
    case kEpiStore: hipLaunchKernelGGL(gemm_reduce<kEpiStore>, rgrid, dim3(256), 0, s, p, ksplit, bn); break;
    case kEpiResidRow: hipLaunchKernelGGL(gemm_reduce<kEpiResidRow>, rgrid, dim3(256), 0, s, p, ksplit, bn); break;
    case kEpiResidF32: hipLaunchKernelGGL(gemm_reduce<kEpiResidF32>, rgrid, dim3(256), 0, s, p, ksplit, bn); break;
    case kEpiRowScale: hipLaunchKernelGGL(gemm_reduce<kEpiRowScale>, rgrid, dim3(256), 0, s, p, ksplit, bn); break;
    case kEpiSwiglu: hipLaunchKernelGGL(gemm_reduce<kEpiSwiglu>, rgrid, dim3(256), 0, s, p, ksplit, bn); break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm_tile(Epilogue epi, const GemmParams& p, int tile, int ksplit, hipStream_t s) {
  if (tile < 0 || tile >= kNumTiles || !tile_ok(p, epi, kTiles[tile]) || ksplit < 1) return hipErrorInvalidValue;
  if (p.lda % 8 || p.ldb % 8) return hipErrorInvalidValue;
  if (ksplit > 1 && (!p.part || (size_t)ksplit * p.M * p.N * sizeof(float) > p.part_bytes))
    return hipErrorInvalidValue;
  GemmParams q = p;
  if (q.n_xcd < 1) q.n_xcd = 1;
  if (q.group_m < 1) q.group_m = 1 << 30;
  return launch_tile_index(tile, epi, q, ksplit, s);
}

// The columns [n1, N) of a product as a product of their own (same rows and
// K): weights, output and residual offset by n1 columns.  SwiGLU counts n1 in
// gate and up rows together (n1 / 2 output columns); other epilogues need a
// single weight block.
static GemmParams columns_from(const GemmParams& p, Epilogue epi, int n1) {
  GemmParams q = p;
  q.N = p.N - n1;
  if (epi == kEpiSwiglu) {
    const int oc = n1 / 2;
    q.b[0] = (const uint16_t*)p.b[0] + (int64_t)oc * p.ldb;
    q.b[1] = (const uint16_t*)p.b[1] + (int64_t)oc * p.ldb;
    q.b[2] = q.b[1];
    q.c = (f16*)p.c + oc;
    return q;
  }
  for (int i = 0; i < 3; ++i) q.b[i] = (const uint16_t*)p.b[0] + (int64_t)n1 * p.ldb;
  q.b_split0 = q.b_split1 = q.N;
  q.c = (float*)p.c + n1;
  if (epi == kEpiResidRow) q.r = (const uint16_t*)p.r + n1;
  if (epi == kEpiResidF32) q.r = (const float*)p.r + n1;
  return q;
}

// A grid of 256 x 256 tiles that takes more than one round and ends in a
// partial one: its whole rounds as 256 x 256 tiles over the first columns (all
// row tiles of each), the remaining columns as 256 x 128 tiles (rate: their
// throughput relative to 256 x 256) in a second launch.  Returns the number of
// 256-wide column tiles of the first launch when that prices cheaper than
// `other` (rounds x tile area / rate of the single-launch choice), else 0.
static int whole_round_columns(const GemmParams& p, int cus, double other, double rate2) {
  const int mt = (p.M + 255) / 256, nt = p.N / 256;
  const long t10 = (long)mt * nt, whole = (t10 / cus) * cus;
  if (p.N % 256 || t10 <= cus || whole == t10 || whole % mt) return 0;
  const int na = (int)(whole / mt);
  const long tail2 = (long)mt * (nt - na) * 2;
  const double cost = (double)(whole / cus) * 65536.0 + (double)((tail2 + cus - 1) / cus) * 32768.0 / rate2;
  return cost < other ? na : 0;
}

hipError_t launch_gemm(DType dt, Epilogue epi, const GemmParams& p0, hipStream_t s) {
  if (p0.M <= 0) return hipSuccess;
  if (dt == kF32) {
    const GemmParams& p = p0;
    const int n_out = epi == kEpiSwiglu ? p.N / 2 : p.N;
    const dim3 grid((n_out + 255) / 256, p.M);
    switch (epi) {
      case kEpiStore: hipLaunchKernelGGL(gemm_f32<kEpiStore>, grid, dim3(256), 0, s, p); break;
      case kEpiResidRow: hipLaunchKernelGGL(gemm_f32<kEpiResidRow>, grid, dim3(256), 0, s, p); break;
      case kEpiResidF32: hipLaunchKernelGGL(gemm_f32<kEpiResidF32>, grid, dim3(256), 0, s, p); break;
      case kEpiRowScale: hipLaunchKernelGGL(gemm_f32<kEpiRowScale>, grid, dim3(256), 0, s, p); break;
      case kEpiSwiglu: hipLaunchKernelGGL(gemm_f32<kEpiSwiglu>, grid, dim3(256), 0, s, p); break;
    }
    return hipGetLastError();
  }
  if (p0.K % 32 || p0.lda % 8 || p0.ldb % 8) return hipErrorInvalidValue;
  GemmParams p = p0;
  const int cus = p.n_cus > 0 ? p.n_cus : 256;
  if (p.n_xcd < 1) p.n_xcd = 1;
  // group of row tiles: the XCD's compute units then cover about a square of
  // tiles (8 row tiles by 4 column tiles with 32 compute units per XCD)
  if (p.group_m < 1) p.group_m = 8;
  auto fits = [&](int ks) { return p.part && (size_t)ks * p.M * p.N * sizeof(float) <= p.part_bytes; };
  // 17..32 rows: the product streams the weights; a 32-row by 128-column tile
  // with four waves, and K split so that the grid has enough workgroups in
  // flight (each slice at least 8 steps of 64).  (Up to 16 rows the one-wave
  // 16-row tiles below measured faster.)
  if (p.M > 16 && p.M <= 32 && tile_ok(p, epi, kTiles[9])) {
    const int tiles = p.N / 128, KT = p.K / 64;
    int ks = 1;
    while (ks < 16 && tiles * ks * 2 <= 4 * cus && KT / (ks * 2) >= 8 && fits(ks * 2)) ks *= 2;
    return launch_tile_index(9, epi, p, ks, s);
  }
  // K of 4096 or more with a few hundred rows (o and down on 129-1024 rows):
  // 256 x 128 tiles with K split re-read the activations and weights half as
  // often as 128 x 64 tiles at the same workgroup count.  As many slices (2-4,
  // of whole 64-deep steps, not necessarily equal) as keep the grid within one
  // round (1024 x 2560 x 9728, 80 tiles: 76 us in three slices against 94 us in
  // two; 1024 x 2560 x 4096: 41 us against 47; 512 x 4096 x 4096, 64 tiles: 38
  // us in four against 41 us for 256 tiles of 128 x 64; 512 x 4096 x 12288: 77
  // us in four against 111 us in two).
  if (epi != kEpiSwiglu && p.M > 128 && p.M <= 1024 && p.K >= 4096 && tile_ok(p, epi, kTiles[2])) {
    const long tiles = (long)((p.M + 255) / 256) * (p.N / 128);
    const int ks = (int)std::min<long>(4, std::max<long>(2, cus / tiles));
    if (p.K % 64 == 0 && p.K / 64 >= 8 * ks && fits(ks)) return launch_tile_index(2, epi, p, ks, s);
  }
  // 33..256 rows, epilogues other than SwiGLU (o, down, the fusion products):
  // the weights stream with few tiles, so 128 x 64 tiles with K split until
  // the grid has a workgroup per compute unit (9B-shaped down on 128 rows:
  // 48 us against 70; o on 256 rows of the 27B shape: 58 us against 71).
  // SwiGLU keeps its wide tiles, which measured faster there.
  if (epi != kEpiSwiglu && p.M > 32 && p.M <= 256 && tile_ok(p, epi, kTiles[3]) && p.part) {
    const long tiles = (long)((p.M + 127) / 128) * (p.N / 64);
    int ks = 2;
    while (ks < 8 && tiles * ks < cus) ks *= 2;
    if (p.K / 64 / ks >= 8 && fits(ks)) return launch_tile_index(3, epi, p, ks, s);
  }
  // The wide tiles, priced by the rounds of workgroups the grid takes on the
  // compute units (a last partial round costs a whole one) times the tile's
  // work over its measured relative rate (2048-8192 rows, fp16 weights).
  auto cheapest = [&](const int* cand, const double* rate, int n) {
    int best = -1;
    double best_cost = 0.0;
    for (int i = 0; i < n; ++i) {
      const TileShape& t = kTiles[cand[i]];
      if (!tile_ok(p, epi, t)) continue;
      const long tiles = (long)((p.M + t.bm - 1) / t.bm) * (p.N / t.bn);
      const double cost = (double)((tiles + cus - 1) / cus) * t.bm * t.bn / rate[i];
      if (best < 0 || cost < best_cost) { best = cand[i]; best_cost = cost; }
    }
    return best;
  };
  // SwiGLU (gate/up) on more than 256 rows, and on 128-256 rows when 256 x 128
  // tiles would fill at least half the compute units (fewer wide tiles would
  // leave most of them idle; the order below then takes smaller ones).  At
  // 1024 x 19456 x 2560 this takes 256 x 128 (608 tiles, 0.140 ms) over
  // 256 x 256 (304 tiles: two rounds, the second nearly empty, 0.154 ms); at
  // 256 x 34816 x 5120 (last-row-only rows of the 27B shape) 256 x 256 in one
  // round of 136 tiles (167 us) over 272 tiles of 256 x 128 (197 us); at
  // 128 x 24576 x 4096, 256 x 128 (82 us) over 128 x 64 (87 us).
  const long tiles2 = (long)((p.M + 255) / 256) * (p.N / 128);
  if (epi == kEpiSwiglu && (p.M > 256 || (p.M >= 128 && 2 * tiles2 >= cus))) {
    static const int cand[4] = {10, 0, 2, 12};
    static const double rate[4] = {1.0, 0.91, 0.87, 0.855};
    const int best = cheapest(cand, rate, 4);
    // (1024 x 19456 x 2560: 124 us against 137 us for 608 tiles of 256 x 128
    // and 149 us for 304 of 256 x 256)
    if (best >= 0 && tile_ok(p, epi, kTiles[10])) {
      const TileShape& tb = kTiles[best];
      const long tb_tiles = (long)((p.M + tb.bm - 1) / tb.bm) * (p.N / tb.bn);
      const int bi = best == 10 ? 0 : best == 0 ? 1 : best == 2 ? 2 : 3;
      const int na = whole_round_columns(p, cus, (double)((tb_tiles + cus - 1) / cus) * tb.bm * tb.bn / rate[bi], 0.87);
      if (na > 0) {
        GemmParams qa = p;
        qa.N = 256 * na;
        const hipError_t e = launch_tile_index(10, epi, qa, 1, s);
        return e != hipSuccess ? e : launch_tile_index(2, epi, columns_from(p, epi, 256 * na), 1, s);
      }
    }
    if (best >= 0) return launch_tile_index(best, epi, p, 1, s);
  }
  // Residual products on more than 1024 rows whose 256 x 128 grid fills the
  // compute units: 8192 x 5120 takes 256 x 160 (four whole rounds; o 0.408 ms,
  // down 1.39 ms) over 256 x 256 (three rounds, the last half empty; 0.413,
  // 1.40) and 256 x 128 (five rounds; 0.428, 1.43).
  // Long K on more than 1024 rows whose 256 x 256 grid fills at most half the
  // compute units: those tiles with K split in two (2048 x 4096 x 12288, down:
  // 201 us against 218 us for 256 tiles of 256 x 128; with K = 4096, o, the
  // split measured slower).
  if (epi != kEpiSwiglu && p.M > 1024 && p.K >= 8192 && tile_ok(p, epi, kTiles[10]) &&
      2 * (long)((p.M + 255) / 256) * (p.N / 256) <= cus && p.K % 128 == 0 && fits(2))
    return launch_tile_index(10, epi, p, 2, s);
  // The mixed plan above applies here too (single weight block): 8192 x 5120
  // as two rounds of 256 x 256 over 4096 columns and one of 256 x 128 over the
  // last 1024 (down 1.22 ms, o 0.369 ms, against 1.34 and 0.389 for 256 x 160).
  if (epi != kEpiSwiglu && p.M > 1024 && tile_ok(p, epi, kTiles[2]) &&
      (long)((p.M + 255) / 256) * (p.N / 128) >= cus) {
    static const int cand[3] = {10, 11, 2};
    static const double rate[3] = {1.0, 0.84, 0.80};
    const int best = cheapest(cand, rate, 3);
    if (best >= 0 && tile_ok(p, epi, kTiles[10]) && p.b_split0 >= p.N) {
      const TileShape& tb = kTiles[best];
      const long tb_tiles = (long)((p.M + tb.bm - 1) / tb.bm) * (p.N / tb.bn);
      const int bi = best == 10 ? 0 : best == 11 ? 1 : 2;
      const int na = whole_round_columns(p, cus, (double)((tb_tiles + cus - 1) / cus) * tb.bm * tb.bn / rate[bi], 0.80);
      if (na > 0) {
        GemmParams qa = p;
        qa.N = qa.b_split0 = qa.b_split1 = 256 * na;
        const hipError_t e = launch_tile_index(10, epi, qa, 1, s);
        return e != hipSuccess ? e : launch_tile_index(2, epi, columns_from(p, epi, 256 * na), 1, s);
      }
    }
    if (best >= 0) return launch_tile_index(best, epi, p, 1, s);
  }
  // First tile (in preference order) that gives at least one workgroup per
  // compute unit, else the valid tile with the most workgroups.
  const int* order = epi == kEpiSwiglu ? kOrderSwiglu : kOrderResid;
  int best = -1;
  long best_tiles = -1;
  for (int i = 0; i < 9; ++i) {
    const int c = order[i];
    if (!tile_ok(p, epi, kTiles[c])) continue;
    const long tiles = (long)((p.M + kTiles[c].bm - 1) / kTiles[c].bm) * (p.N / kTiles[c].bn);
    if (tiles >= cus) { best = c; break; }
    if (tiles > best_tiles) { best_tiles = tiles; best = c; }
  }
  return launch_tile_index(best, epi, p, 1, s);
}

}  // namespace sp
