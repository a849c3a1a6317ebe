// Split attention of the k soft queries over the cached prefix (Sec. 3.3,
// Eq. 1-3).
//
// Rows of a KV head: its k*G soft queries (row r = j*G + h%G for soft row j and
// query head h = g*G + h%G).  Split s covers cache tokens [s*split_len,
// min(N_b, (s+1)*split_len)).  Each split keeps an online softmax per row
// (running max m in log2 units, running sum l, unnormalised output O) and
// writes it as a partial (m, l and, on the bf16 path, O / l in fp16); the
// merge (merge.hip) adds the soft keys and combines the partials.
//
// bf16 path: bf16 KV cache, bf16 MFMA operands, fp32 accumulation.  The two
// operands the kernel itself rounds, the queries and the probabilities, are
// carried as hi + lo bf16 pairs (x = hi + lo to ~16 bits), so every product
// is K*Q_hi + K*Q_lo and P_hi*V + P_lo*V with K and V exact as stored.
// One workgroup per (sequence, KV head, query group, split) with one wave per
// 16-row query tile.  The split's tokens are consumed in units of 32 (two
// 16-token halves, each inside one block):
//   * the workgroup loads each unit's K and V tiles straight into LDS (16-byte
//     direct loads, streaming), two units ahead, through three LDS stages; in
//     a tail unit, V slots past the end are zeroed after landing (their bytes
//     may be anything, NaN included);
//   * every wave reads its fragments from LDS and runs its query tile:
//     S^T = K Q^T on v_mfma_f32_16x16x32_bf16, so that lane (li, la) ends up
//     with 8 consecutive tokens of query li: the A operand of
//     v_mfma_f32_16x16x32_bf16 for O += P V (P never goes through LDS); the B
//     operand is V[those 8 tokens][16nt + li], 16 contiguous LDS bytes.
// Online softmax in log2 units with a lazy reference max (see kRescaleLog2).
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace sp {
namespace {

__device__ __forceinline__ int64_t phys_block(const AttnParams& p, int b, int t) {
  const int lb = t >> p.bs_log2;
  return p.block_table ? (int64_t)p.block_table[(int64_t)b * p.mbps + lb]
                       : (int64_t)b * p.mbps + lb;
}

// A row's reference max moves only when a score exceeds it by more than this
// (log2 units), so probabilities stay below 2^8 between moves.
constexpr float kRescaleLog2 = 8.0f;

// The wave's running softmax state for its 16 query rows.  F16: the fp16
// variant (single fp16 products on K and V converted to fp16 in LDS).
template <int HD, bool F16>
struct RowState {
  static constexpr int NC = HD / 32, NT = HD / 16;
  bf16x8 qh[NC], ql[NC];  // Q[row li][8 (la*NC + c) .. +7], hi and lo parts (bf16 products)
  f16x8 q16[NC];          // the same rows rounded to fp16 (fp16 products)
  f32x4 o[NT];            // O[row 4la + r][16nt + li], unnormalised
  float m, l;             // reference max of row li (log2 units); this lane's part of its sum
};

// One 32-token unit for one wave, in two phases.  qk_unit: kf[h][c] =
// K[token pi_h(li)][8 (la*NC + c) ..] (the unit layout below); score i of the
// lane (i = 4h + r) is token 8la + i for query li.  The accumulators start at
// -m (the row's reference max), so the scores come out as s - m, except in the
// first unit of a split (FIRST), whose reference is still the -1e30 start
// value: it takes the raw scores.  softmax_pv_unit: vf[nt] =
// V[tokens 8la..8la+7][16nt + li]; keys at or past `limit` are masked.
template <int HD, bool FIRST, bool F16>
__device__ __forceinline__ void qk_unit(const RowState<HD, F16>& st, const u32x4 (&kf)[2][HD / 32],
                                        f32x4& s0, f32x4& s1) {
  constexpr int NC = HD / 32;
  const float init = FIRST ? 0.f : -st.m;
  s0 = f32x4{init, init, init, init};
  s1 = s0;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    if constexpr (F16) {
      s0 = mfma16x16x32(__builtin_bit_cast(f16x8, kf[0][c]), st.q16[c], s0);
      s1 = mfma16x16x32(__builtin_bit_cast(f16x8, kf[1][c]), st.q16[c], s1);
    } else {
      const bf16x8 k0 = __builtin_bit_cast(bf16x8, kf[0][c]), k1 = __builtin_bit_cast(bf16x8, kf[1][c]);
      s0 = mfma16x16x32_bf16(k0, st.qh[c], s0);
      s1 = mfma16x16x32_bf16(k1, st.qh[c], s1);
      s0 = mfma16x16x32_bf16(k0, st.ql[c], s0);
      s1 = mfma16x16x32_bf16(k1, st.ql[c], s1);
    }
  }
}

// p = hi + lo for two values at a time: hi = bf16(p) (round to nearest even),
// lo = bf16(p - hi); both pairs packed as the MFMA operand expects.
__device__ __forceinline__ void split_pair(float p0, float p1, uint32_t& hi, uint32_t& lo) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
  hi = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{p0, p1}, bf16x2v));
  const float h0 = __builtin_bit_cast(float, hi << 16), h1 = __builtin_bit_cast(float, hi & 0xffff0000u);
  lo = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{p0 - h0, p1 - h1}, bf16x2v));
}

template <int HD, bool FIRST, bool F16>
__device__ __forceinline__ void softmax_pv_unit(RowState<HD, F16>& st, f32x4 s0, f32x4 s1,
                                                const u32x4 (&vf)[HD / 16], int la, int limit) {
  constexpr int NT = HD / 16;
  // sc = s - m, or s in the first unit
  float sc[8] = {s0[0], s0[1], s0[2], s0[3], s1[0], s1[1], s1[2], s1[3]};
  if (limit < 32) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (8 * la + i >= limit) sc[i] = -INFINITY;
  }
  float lmax = fmaxf(fmaxf(sc[0], sc[1]), sc[2]);
  lmax = fmaxf(fmaxf(lmax, sc[3]), sc[4]);
  lmax = fmaxf(fmaxf(lmax, sc[5]), sc[6]);
  lmax = fmaxf(lmax, sc[7]);
  // Lazy reference max: p = 2^(s - m) with m the row's reference, which only
  // moves (with the cross-lane reduction and the rescale of l and O) when some
  // score exceeds it by more than kRescaleLog2.
  const float excess = FIRST ? lmax - st.m : lmax;
  if (__any(excess > kRescaleLog2)) {
    float rm = fmaxf(lmax, __shfl_xor(lmax, 16));  // the row's max (shifted or raw)
    rm = fmaxf(rm, __shfl_xor(rm, 32));
    float alpha;
    if (!FIRST) {
      const float delta = fmaxf(rm, 0.f);  // the reference moves up by delta
      alpha = fast_exp2(-delta);
      st.m += delta;
#pragma unroll
      for (int i = 0; i < 8; ++i) sc[i] -= delta;
    } else {
      const float mn = fmaxf(st.m, rm);
      alpha = fast_exp2(st.m - mn);
      st.m = mn;
#pragma unroll
      for (int i = 0; i < 8; ++i) sc[i] -= mn;
    }
    st.l *= alpha;
    // O rows held by this lane are queries 4la + r; their factors live in lanes 4la + r.
    float ar[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) ar[r] = __shfl(alpha, 4 * la + r);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r) st.o[nt][r] *= ar[r];
  } else if (FIRST) {
#pragma unroll
    for (int i = 0; i < 8; ++i) sc[i] -= st.m;
  }
  float pv[8];
  float ps = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    pv[i] = fast_exp2(sc[i]);
    ps += pv[i];
  }
  st.l += ps;
  if constexpr (F16) {
    // p < 2^8 between reference moves: fp16 (round to nearest even) keeps 11 bits
    f16x8 p16;
#pragma unroll
    for (int i = 0; i < 8; ++i) p16[i] = (f16)pv[i];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) st.o[nt] = mfma16x16x32(p16, __builtin_bit_cast(f16x8, vf[nt]), st.o[nt]);
  } else {
    uint32_t hw[4], lw[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) split_pair(pv[2 * q], pv[2 * q + 1], hw[q], lw[q]);
    const bf16x8 ph = __builtin_bit_cast(bf16x8, u32x4{hw[0], hw[1], hw[2], hw[3]});
    const bf16x8 pl = __builtin_bit_cast(bf16x8, u32x4{lw[0], lw[1], lw[2], lw[3]});
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const bf16x8 v = __builtin_bit_cast(bf16x8, vf[nt]);
      st.o[nt] = mfma16x16x32_bf16(ph, v, st.o[nt]);
      st.o[nt] = mfma16x16x32_bf16(pl, v, st.o[nt]);
    }
  }
}

// LDS image of a 32-token unit, in 16-byte pieces.  Token T of the unit lies
// in half T >> 4 (16 tokens inside one block, slots t = T & 15).  The QK
// product of half-MFMA h (h = 0, 1) takes, as its row m, token
//   pi_h(m) = 8 (m >> 2) + 4 h + (m & 3),
// so that lane (li, la) receives scores of tokens 8 la + 4 h + r, i.e. tokens
// 8 la .. 8 la + 7 over both half-MFMAs: exactly its A operand of the PV MFMA.
// Pieces are grouped by half, so that each 64-piece wave-instruction of the
// direct loads reads from one block:
//   K half hh: piece hh * KHP + c8 * 16 + t = K[16 hh + t][8 c8 .. 8 c8 + 7]
//   V half hh: piece VB + hh * 2 HD + (2 nt + e) * 16 + li
//                    = V[16 hh + 8 e .. 16 hh + 8 e + 7][16 nt + li]
// A K fragment read (16 lanes: tokens pi_h(0..15), 8 from each half) then
// covers 16 distinct 16-byte bank groups thanks to the 4-piece pad of the
// second K half; a V fragment read is 256 contiguous bytes per 16 lanes.
template <int HD>
struct UnitLayout {
  static constexpr int NI = HD / 8;           // wave-instructions (64 pieces each) per unit
  static constexpr int IPG = HD / 32;         // wave-instructions per (tensor, half) group
  static constexpr int KHP = 2 * HD + 4;      // K half pitch (pieces), padded
  static constexpr int VB = KHP + 2 * HD;     // first V piece
  static constexpr int PIECES = VB + 4 * HD;  // pieces per stage
  // first piece of group gi (0: K half 0, 1: K half 1, 2: V half 0, 3: V half 1)
  static constexpr __device__ int group_base(int gi) {
    return gi == 0 ? 0 : gi == 1 ? KHP : gi == 2 ? VB : VB + 2 * HD;
  }
  static __device__ __forceinline__ int k_piece(int h, int c8, int li) {
    const int tk = 8 * (li >> 2) + 4 * h + (li & 3);
    return (tk >> 4) * KHP + c8 * 16 + (tk & 15);
  }
  static __device__ __forceinline__ int v_piece(int nt, int li, int la) {
    return VB + (la >> 1) * 2 * HD + (2 * nt + (la & 1)) * 16 + li;
  }
};

// The split's physical block ids live in LDS in a rolling table of two windows
// of kIdWin logical blocks (window w in slot w & 1).
constexpr int kIdWin = 512;

// Direct global -> LDS load of 4 bytes per lane (lane l's at wave_dst + 4 l);
// waited for like ld16_to_lds.
__device__ __forceinline__ void ld4_to_lds(const void* base, uint32_t lane_off, int* wave_dst) {
  const uint32_t lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) int*)wave_dst;
  asm volatile("global_load_lds_dword %0, %1" : : "v"(lane_off), "s"(base), "{m0}"(lds) : "memory");
}

// Zero the V values of tokens at or past `limit` in a staged tail unit (the
// bytes there may be anything, NaN included, and P V would carry 0 * NaN).
template <int HD, int W>
__device__ __forceinline__ void zero_tail(u32x4* sb, int limit, int tid) {
  u32x4* v = sb + UnitLayout<HD>::VB;
  for (int q = tid; q < 4 * HD; q += 64 * W) {
    const int tk0 = 16 * (q / (2 * HD)) + 8 * ((q >> 4) & 1);  // first of the piece's 8 tokens
    if (tk0 + 8 > limit) {
      u32x4 x = v[q];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int keep = limit - (tk0 + 2 * w);
        x[w] &= keep >= 2 ? 0xffffffffu : (keep == 1 ? 0x0000ffffu : 0u);
      }
      v[q] = x;
    }
  }
}

// Wait until at most k units of PPL loads each remain in flight (k <= K).
template <int PPL, int K>
__device__ __forceinline__ void wait_units_le(int k) {
  if constexpr (K == 0) {
    wait_vmcnt<0>();
  } else {
    if (k >= K) wait_vmcnt<K * PPL>();
    else wait_units_le<PPL, K - 1>(k);
  }
}

// A wave's fragments of a staged unit, then the unit's softmax and products
// for each of the wave's ntw (<= TPW) query tiles: every K and V fragment read
// from LDS serves all of them.
template <int HD, bool FIRST, bool F16, int TPW>
__device__ __forceinline__ void compute_unit(RowState<HD, F16> (&st)[TPW], int ntw, const u32x4* sb, int limit,
                                             int li, int la) {
  constexpr int NC = HD / 32, NT = HD / 16;
  f32x4 s0[TPW], s1[TPW];
  {
    u32x4 kf[2][NC];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int c = 0; c < NC; ++c) kf[h][c] = sb[UnitLayout<HD>::k_piece(h, la * NC + c, li)];
#pragma unroll
    for (int t = 0; t < TPW; ++t)
      if (t < ntw) qk_unit<HD, FIRST, F16>(st[t], kf, s0[t], s1[t]);
  }
  // V fragments are read only once the QK products are issued, into the
  // registers the K fragments held.
  __builtin_amdgcn_sched_barrier(0);
  u32x4 vf[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) vf[nt] = sb[UnitLayout<HD>::v_piece(nt, li, la)];
#pragma unroll
  for (int t = 0; t < TPW; ++t)
    if (t < ntw) softmax_pv_unit<HD, FIRST, F16>(st[t], s0[t], s1[t], vf, la, limit);
}

// fp16 variant: convert a landed unit's K and V tiles in LDS from bf16 to fp16
// in place (exact for magnitudes in fp16's normal range), once for all the
// workgroup's waves, zeroing V slots at or past `limit` (they may hold NaN).
template <int HD, int W>
__device__ __forceinline__ void convert_unit(u32x4* sb, int limit, int tid) {
  using L = UnitLayout<HD>;
  for (int q = tid; q < 8 * HD; q += 64 * W) {
    const bool is_v = q >= 4 * HD;
    const int piece = is_v ? L::VB + (q - 4 * HD) : (q / (2 * HD)) * L::KHP + q % (2 * HD);
    u32x4 x = bf16x8_to_f16x8(sb[piece]);
    if (is_v && limit < 32) {
      const int qv = q - 4 * HD;
      const int tk0 = 16 * (qv / (2 * HD)) + 8 * ((qv >> 4) & 1);  // first of the piece's 8 tokens
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int keep = limit - (tk0 + 2 * w);
        x[w] &= keep >= 2 ? 0xffffffffu : (keep == 1 ? 0x0000ffffu : 0u);
      }
    }
    sb[piece] = x;
  }
}

// W waves per workgroup, each with one 16-row query tile, or with TPW > 1 an
// even share of the group's n_tiles tiles (every K/V fragment read from LDS
// then serves all of a wave's tiles), NS LDS stages (3 here).  bf16 products:
// unit u is computed from stage u % NS while units u + 1 .. u + NS - 1 are in
// flight.  F16: at step u the workgroup converts unit u + 1 to fp16 in LDS
// while it computes unit u, units u + 2 .. u + NS - 1 in flight, so each K/V
// element is converted once for all W waves and every product is a single
// fp16 MFMA (half the matrix-core work of the hi + lo bf16 pairs).
template <int HD, int W, bool ROT, bool F16, int NS, int TPW>
__global__ __launch_bounds__(W * 64) void attn_split_bf16(const AttnParams p) {
  constexpr int NC = HD / 32, NT = HD / 16;
  constexpr int NI = UnitLayout<HD>::NI;
  constexpr int PPL = (NI + W - 1) / W;  // wave-instructions per wave per unit
  constexpr int D = NS - 1;              // issue distance in units
  static_assert(W <= 2 * NI, "a wave must have at least one distinct instruction slot");
  static_assert(NS >= 3 && (NS - 2) * PPL < 64, "stages");
  __shared__ u32x4 stage[NS][UnitLayout<HD>::PIECES];
  __shared__ int blk_ids[2][kIdWin];  // physical blocks of the split (rolling windows)

  const int tid = threadIdx.x, lane = tid & 63, li = lane & 15, la = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  __builtin_assume(tid < 64 * W);
  __builtin_assume(wave >= 0 && wave < W);
  // Grid (KV head + n_kv * query group, split, sequence slot): workgroups are dealt
  // to the 8 XCDs round-robin in linear order, so with n_kv a multiple of 8
  // each XCD takes whole KV heads (the same work for every head), and the
  // query groups of one (sequence, KV head, split), which read the same K/V,
  // run on one XCD at about the same time.  With the split index fastest,
  // the splits past the end of short sequences (which exit at once) would all
  // fall on the same XCDs.
  const int g = blockIdx.x % p.n_kv, qg = blockIdx.x / p.n_kv;
  // Work item of this slot: from the work list (longest items first, so the
  // short ones fill the end of the launch, and no slot lands on a split past
  // the end of its sequence), else (sequence z, split y).
  int b = blockIdx.z, s = blockIdx.y;
  if (p.items) {
    const int L = blockIdx.y + blockIdx.z * gridDim.y;
    if (L >= *p.n_items) return;
    const int2 it = p.items[L];
    b = __builtin_amdgcn_readfirstlane(it.x);
    s = __builtin_amdgcn_readfirstlane(it.y);
  }
  if (p.err && *p.err) return;
  const int n = clamp_len(p.seq_lens, b, p.max_seq_len);
  const int t0 = s * p.split_len;
  if (s > 0 && t0 >= n) return;  // (only without the work list)
  const int t1 = min(n, t0 + p.split_len);
  // this wave's query tiles: [tb, tb + ntw) of the group's n_tiles (one each
  // when TPW = 1, else an even share of at most TPW)
  const int tb = TPW == 1 ? wave : wave * p.n_tiles / W;
  const int ntw = TPW == 1 ? 1 : (wave + 1) * p.n_tiles / W - tb;
  const int row0 = (qg * p.n_tiles + tb) * 16;  // first of this wave's rows in the KV head
  const int bs = 1 << p.bs_log2;

  RowState<HD, F16> st[TPW];
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) st[t].o[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    st[t].m = kNegBig;
    st[t].l = 0.f;
    if (t >= ntw) continue;
    const int64_t qo = (((int64_t)b * p.n_kv + g) * p.r_alloc + row0 + 16 * t + li) * HD;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      st[t].qh[c] = __builtin_bit_cast(bf16x8, ld16v((const bf16*)p.q + qo + 8 * (la * NC + c)));
      st[t].ql[c] = __builtin_bit_cast(bf16x8, ld16v((const bf16*)p.q_lo + qo + 8 * (la * NC + c)));
      if constexpr (F16)
#pragma unroll
        for (int i = 0; i < 8; ++i) st[t].q16[c][i] = (f16)((float)st[t].qh[c][i] + (float)st[t].ql[c][i]);
    }
  }

  const int nunits = (t1 - t0 + 31) >> 5;   // 0 when the split has no cache tokens
  if (nunits > 0) {
    const bf16* kbase = (const bf16*)p.k_base + (int64_t)g * p.k_sh;
    const bf16* vbase = (const bf16*)p.v_base + (int64_t)g * p.v_sh;
    // Physical block of logical block lb0 + rel: windows 0 and 1 are read now;
    // window w + 1 is loaded (direct loads into LDS, one wave-instruction per
    // 64 ids) when issuing enters window w, kIdWin blocks before it is needed.
    // A unit's two halves always fall in one window (rel of its first half is
    // even: t0 is a multiple of 32 tokens, blocks hold >= 16).
    const int lb0 = t0 >> p.bs_log2;
    const int nlb = ((t1 - 1) >> p.bs_log2) - lb0 + 1;
    const int* bt_row = p.block_table ? p.block_table + (int64_t)b * p.mbps + lb0 : nullptr;
    if (bt_row)
      for (int i = tid; i < min(nlb, 2 * kIdWin); i += 64 * W) blk_ids[i / kIdWin][i % kIdWin] = bt_row[i];
    // Physical blocks of logical blocks lb0 + ra and lb0 + rb; both table reads
    // are issued before either is used (one LDS round trip, not two).
    auto phys2 = [&](int ra, int rb, int64_t& pa, int64_t& pb) __attribute__((always_inline)) {
      if (bt_row) {
        const unsigned ua = (unsigned)ra, ub = (unsigned)rb;
        const int ia = blk_ids[(ua / kIdWin) & 1][ua % kIdWin];
        const int ib = blk_ids[(ub / kIdWin) & 1][ub % kIdWin];
        pa = (int64_t)__builtin_amdgcn_readfirstlane(ia);
        pb = (int64_t)__builtin_amdgcn_readfirstlane(ib);
      } else {
        pa = (int64_t)b * p.mbps + lb0 + ra;
        pb = (int64_t)b * p.mbps + lb0 + rb;
      }
    };
    auto load_window = [&](int w) __attribute__((always_inline)) {
      for (int j = wave; j < kIdWin / 64; j += W) {
        const int rel = min(w * kIdWin + j * 64 + lane, nlb - 1);  // past the end: re-read the last id
        ld4_to_lds(bt_row, (uint32_t)rel * 4u, &blk_ids[w & 1][j * 64]);
      }
    };
    // Nothing the compiler tracks stays in flight past this point (the Q loads
    // included), so it never waits on the vector-memory counter inside the loop,
    // where the counter also holds the direct-to-LDS loads.
    wait_vmcnt<0>();
    lds_barrier();
    // This wave's wave-instructions: slots j*W + wave (mod NI, so a wave count
    // that does not divide NI re-issues a few slots; the copies carry the same
    // bytes).  Slot sl reads group gi = sl / IPG (K or V of one half); the lane's
    // byte offset inside that half's tile and the slot's place in the stage do
    // not change from unit to unit, only the four group bases do.  When W
    // divides IPG, the group of each j is a compile-time constant.
    using L = UnitLayout<HD>;
    constexpr bool kStaticGroups = L::IPG % W == 0;
    uint32_t lane_off[PPL];
    int gsel[PPL], lds_piece[PPL];
#pragma unroll
    for (int j = 0; j < PPL; ++j) {
      const int slot = (j * W + wave) % NI;
      gsel[j] = kStaticGroups ? j * W / L::IPG : slot / L::IPG;
      lds_piece[j] = L::group_base(gsel[j]) + (slot % L::IPG) * 64;
      const int q = (slot % L::IPG) * 64 + lane;  // piece inside its group
      if (gsel[j] < 2)
        lane_off[j] = (uint32_t)(((q >> 4) * bs + (q & 15)) * 16);                       // K: c8, t
      else
        lane_off[j] = (uint32_t)((16 * (q >> 5) + (q & 15)) * bs * 2 + ((q >> 4) & 1) * 16);  // V: i, e
    }
    // Unit u: halves start at t0 + 32u and t0 + 32u + 16; a half whose first
    // token is past the end re-reads the first half (then masked), so every
    // address lies in a block the sequence owns.
    // Loads are non-temporal (read once), except V in blocks of more than 32
    // tokens: a V row (one head dim) then spans more than a unit, so a unit
    // reads 64 bytes of a 128-byte line and the next unit the other 64, which
    // must still be in L2 (4096-token blocks: 166 us against 212 with the hint).
    const bool v_stream = p.bs_log2 <= 5;
    auto issue = [&](int u, int buf) __attribute__((always_inline)) {
      const int ta = t0 + 32 * u;
      const int tb = ta + 16 < t1 ? ta + 16 : ta;
      int64_t ba, bb;
      phys2((ta >> p.bs_log2) - lb0, (tb >> p.bs_log2) - lb0, ba, bb);
      const int sa = ta & (bs - 1), sbb = tb & (bs - 1);
      const bf16* g0 = kbase + ba * p.k_sb + sa * 8;
      const bf16* g1 = kbase + bb * p.k_sb + sbb * 8;
      const bf16* g2 = vbase + ba * p.v_sb + sa;
      const bf16* g3 = vbase + bb * p.v_sb + sbb;
#pragma unroll
      for (int j = 0; j < PPL; ++j) {
        const int gi = gsel[j];
        const bf16* gb = gi == 0 ? g0 : gi == 1 ? g1 : gi == 2 ? g2 : g3;
        if (gi < 2 || v_stream)
          ld16_to_lds(gb, lane_off[j], &stage[buf][lds_piece[j]]);
        else
          ld16_to_lds<false>(gb, lane_off[j], &stage[buf][lds_piece[j]]);
      }
    };
    const int last = nunits - 1;
    // wait until at most k (0 <= k <= NS - 2) units of this wave's loads remain in flight
    auto wait_units = [&](int k) __attribute__((always_inline)) { wait_units_le<PPL, NS - 2>(k); };
#pragma unroll
    for (int v = 0; v < D; ++v)
      if (v <= last) issue(v, v);
    if constexpr (F16) {
      // unit 0 converted before the loop (its conversion is published by step 0's barrier)
      wait_units(min(D - 1, last));
      lds_barrier();
      convert_unit<HD, W>(stage[0], t1 - t0, tid);
    }
    int buf = 0;
    // One unit: wait for its loads, publish them, issue unit u + 2, compute.
    // The first unit is peeled (raw scores; see qk_unit).
    // Co-resident workgroups share a compute unit's wave arbiter, which favours
    // the oldest waves: in a grid of one round (every workgroup resident from
    // the start), the workgroups of a compute unit would end one after another
    // in dispatch order and the launch on a tail at one or two per compute
    // unit.  There (ROT) their wave priorities rotate with the 100 MHz
    // real-time counter (every 2^12 ticks, 41 us): a workgroup's dispatch pass
    // (one workgroup per compute unit per pass) sets its phase, so the
    // workgroups of one compute unit take turns at each priority level.
    // Timing only: what each workgroup computes does not change.
    const int rot_phase =
        (int)(((blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z)) / p.num_cus) % 3);
    auto rotate_priority = [&]() __attribute__((always_inline)) {
      const int ep = (int)((__builtin_amdgcn_s_memrealtime() >> 12) % 3);
      const int pr = __builtin_amdgcn_readfirstlane((rot_phase + ep) % 3);
      if (pr == 0) __builtin_amdgcn_s_setprio(0);
      else if (pr == 1) __builtin_amdgcn_s_setprio(1);
      else __builtin_amdgcn_s_setprio(2);
    };
    // Entering window w >= 1 of the block ids when issuing unit v: load window
    // w + 1 (it replaces window w - 1, which no later issue reads).  Loads issued
    // after the unit's only make the next vmcnt waits stricter.
    auto next_window = [&](int v) __attribute__((always_inline)) {
      const int w = (((t0 + 32 * v) >> p.bs_log2) - lb0) / kIdWin;
      const int wprev = (((t0 + 32 * (v - 1)) >> p.bs_log2) - lb0) / kIdWin;
      if (bt_row && w != wprev && (w + 1) * kIdWin < nlb) load_window(w + 1);
    };
    auto step = [&](int u, auto first) __attribute__((always_inline)) {
      const int limit = t1 - (t0 + 32 * u);
      // units issued so far: 0 .. min(u + D - 1, last)
      const int issued = min(u + D - 1, last);
      if constexpr (!F16) {
        // this wave's loads of unit u are done once at most those of the later issued units remain
        wait_units(issued - u);
        // every wave's loads of unit u have landed and every wave is done with unit u - 1
        lds_barrier();
        if constexpr (ROT)
          if ((u & 3) == 0) rotate_priority();
        if (limit < 32) {
          zero_tail<HD, W>(stage[buf], limit, tid);
          lds_barrier();
        }
      } else {
        // this wave's loads of unit u + 1 are done once at most those of the later issued units remain
        wait_units(max(issued - u - 1, 0));
        // every wave's loads of unit u + 1 have landed, unit u's conversion is
        // visible, every wave is done with unit u - 1
        lds_barrier();
        if constexpr (ROT)
          if ((u & 3) == 0) rotate_priority();
      }
      // unit u + D into the stage of unit u - 1
      if (u + D <= last) {
        issue(u + D, buf == 0 ? NS - 1 : buf - 1);
        next_window(u + D);
      }
      if constexpr (F16)
        if (u + 1 <= last) convert_unit<HD, W>(stage[buf == NS - 1 ? 0 : buf + 1], limit - 32, tid);
      compute_unit<HD, decltype(first)::value, F16, TPW>(st, ntw, stage[buf], limit, li, la);
      buf = buf == NS - 1 ? 0 : buf + 1;
    };
    step(0, std::true_type{});
    for (int u = 1; u < nunits; ++u) step(u, std::false_type{});
  }

#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    if (t >= ntw) continue;
    const int64_t prow = (((int64_t)b * p.n_kv + g) * p.max_splits + s) * p.r_alloc + row0 + 16 * t;
    float lt = st[t].l;
    lt += __shfl_xor(lt, 16);
    lt += __shfl_xor(lt, 32);
    if (la == 0) p.ml_part[prow + li] = make_float2(st[t].m, lt);
    // O / l in fp16: a convex combination of the split's values, so within fp16
    // whenever V is (the merge weights it by l again); lane (li, la) holds rows
    // 4la + r, whose sums sit in lanes 4la + r
    float inv[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float lr = __shfl(lt, 4 * la + r);
      inv[r] = lr > 0.f ? 1.0f / lr : 0.f;
    }
    f16* op = (f16*)p.o_part;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r) op[(prow + 4 * la + r) * HD + 16 * nt + li] = (f16)(st[t].o[nt][r] * inv[r]);
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
  if (s > 0 && t0 >= n) return;  // (only without the work list)
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

  // cache tokens [c0, c0 + TT)
  auto run_chunk = [&](int c0) {
    for (int idx = tid; idx < TT * HD; idx += 256) {
      const int t = idx / HD, i = idx % HD, tok = c0 + t;
      float kv = 0.f, vv = 0.f;
      if (tok < t1) {
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
      const int r = idx / TT, t = idx % TT;
      float acc = 0.f;
      for (int i = 0; i < HD; ++i) acc += qs[r][i] * ks[t][i];
      ps[r][t] = c0 + t < t1 ? acc : -INFINITY;
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

  for (int c0 = t0; c0 < t1; c0 += TT) run_chunk(c0);

  const int64_t prow = (((int64_t)b * p.n_kv + g) * p.max_splits + s) * p.r_alloc;
  if (tid < R) p.ml_part[prow + tid] = make_float2(m_s[tid], l_s[tid]);
#pragma unroll
  for (int u = 0; u < OPT; ++u) {
    const int idx = tid + 256 * u;
    const int r = idx / HD, i = idx % HD;
    if (r < R) ((float*)p.o_part)[(prow + r) * HD + i] = oacc[u];
  }
}

// One workgroup of 1024 threads: the work list (see launch_work_list).  Full
// splits: an exclusive scan of (splits - 1) per sequence, 1024 sequences at a
// time; last splits: the rank of each by (tokens descending, sequence), the
// candidates staged 1024 at a time in LDS.
__global__ __launch_bounds__(1024) void work_list(const int* seq_lens, int batch, int max_seq_len, int split_len,
                                                  int2* items, int* count) {
  __shared__ __align__(16) int scan[1024];
  __shared__ int carry;
  const int tid = threadIdx.x;
  auto splits = [&](int b) { const int n = clamp_len(seq_lens, b, max_seq_len); return n > 0 ? (n + split_len - 1) / split_len : 1; };
  auto last_tokens = [&](int b) { const int n = clamp_len(seq_lens, b, max_seq_len); return n - (splits(b) - 1) * split_len; };
  if (tid == 0) carry = 0;
  __syncthreads();
  for (int b0 = 0; b0 < batch; b0 += 1024) {
    const int b = b0 + tid;
    const int nf = b < batch ? splits(b) - 1 : 0;
    scan[tid] = nf;
    __syncthreads();
    for (int o = 1; o < 1024; o <<= 1) {
      const int v = tid >= o ? scan[tid - o] : 0;
      __syncthreads();
      scan[tid] += v;
      __syncthreads();
    }
    const int off = carry + scan[tid] - nf;
    for (int sp = 0; sp < nf; ++sp) items[off + sp] = make_int2(b, sp);
    __syncthreads();
    if (tid == 1023) carry += scan[1023];
    __syncthreads();
  }
  const int full = carry;
  for (int b0 = 0; b0 < batch; b0 += 1024) {
    const int b = b0 + tid;
    const int rb = b < batch ? last_tokens(b) : 0;
    int rank = 0;
    for (int o0 = 0; o0 < batch; o0 += 1024) {
      __syncthreads();
      scan[tid] = o0 + tid < batch ? last_tokens(o0 + tid) : -1;  // -1: no sequence (ranks below all)
      __syncthreads();
      // four counts per 16-byte LDS read (the slots past the batch hold -1)
      const int m4 = (min(1024, batch - o0) + 3) / 4;
      const int4* s4 = (const int4*)scan;
#pragma unroll 4
      for (int q = 0; q < m4; ++q) {
        const int4 r = s4[q];
        const int j = o0 + 4 * q;
        rank += (r.x > rb) || (r.x == rb && j < b);
        rank += (r.y > rb) || (r.y == rb && j + 1 < b);
        rank += (r.z > rb) || (r.z == rb && j + 2 < b);
        rank += (r.w > rb) || (r.w == rb && j + 3 < b);
      }
    }
    if (b < batch) items[full + rank] = make_int2(b, splits(b) - 1);
  }
  if (tid == 0) count[0] = full + batch;
}

}  // namespace

hipError_t launch_work_list(const int* seq_lens, int batch, int max_seq_len, int split_len, int2* items, int* count,
                            hipStream_t s) {
  if (batch <= 0) return hipSuccess;
  if (split_len < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(work_list, dim3(1), dim3(1024), 0, s, seq_lens, batch, max_seq_len, split_len, items, count);
  return hipGetLastError();
}

hipError_t launch_attention_bf16(const AttnParams& p, int hd, int waves, int batch, hipStream_t s) {
  const bool f16 = p.f16;
  const int stages = p.stages;
  // query tiles per wave (the group's n_tiles over its waves)
  const int tpw = (p.n_tiles + waves - 1) / waves;
  if (p.n_tiles < waves || tpw > 4) return hipErrorInvalidValue;
  if (p.bs_log2 < 4 || p.split_len % 32) return hipErrorInvalidValue;
  const dim3 grid(p.n_kv * p.n_qgroups, p.max_splits, batch);
  if (p.n_qgroups * p.n_tiles * 16 != p.r_alloc) return hipErrorInvalidValue;
  // Rotating priorities pays where several multi-wave workgroups share each
  // compute unit for the whole launch: a grid of at most one round (long
  // uniform batches: 83% of HBM peak against 78%).  Grids of many rounds
  // refill compute units as workgroups end, and one-wave workgroups do not
  // stagger; there the clock reads only cost time (2-5% measured).
  if (p.num_cus < 1) return hipErrorInvalidValue;
  const int per_cu = attn_wgs_per_cu(hd, waves, tpw);
  const bool rot = waves >= 2 && per_cu >= 2 && (int64_t)grid.x * grid.y * grid.z <= (int64_t)p.num_cus * per_cu;
#define SP_ATTN_CASE(HD_, W_)                                                                 \
  if (!f16 && hd == HD_ && waves == W_ && tpw == 1 && stages == 3) {                          \
    hipLaunchKernelGGL((attn_split_bf16<HD_, W_, false, false, 3, 1>), grid, dim3(64 * W_), 0, s, p); \
    return hipGetLastError();                                                                 \
  }
#define SP_ATTN_CASE_ROT(HD_, W_)                                                             \
  if (!f16 && hd == HD_ && waves == W_ && tpw == 1 && stages == 3) {                          \
    if (rot) hipLaunchKernelGGL((attn_split_bf16<HD_, W_, true, false, 3, 1>), grid, dim3(64 * W_), 0, s, p); \
    else hipLaunchKernelGGL((attn_split_bf16<HD_, W_, false, false, 3, 1>), grid, dim3(64 * W_), 0, s, p);    \
    return hipGetLastError();                                                                 \
  }
#define SP_ATTN_CASE_MULTI(HD_, W_, TPW_)                                                     \
  if (hd == HD_ && waves == W_ && tpw == TPW_ && stages == 3) {                              \
    if (f16) hipLaunchKernelGGL((attn_split_bf16<HD_, W_, false, true, 3, TPW_>), grid, dim3(64 * W_), 0, s, p); \
    else hipLaunchKernelGGL((attn_split_bf16<HD_, W_, false, false, 3, TPW_>), grid, dim3(64 * W_), 0, s, p);    \
    return hipGetLastError();                                                                 \
  }
  // several query tiles per wave (8-16 tiles per group on 4 waves; fp16 products)
  SP_ATTN_CASE_MULTI(128, 4, 2) SP_ATTN_CASE_MULTI(128, 4, 3)
  SP_ATTN_CASE_MULTI(64, 4, 2) SP_ATTN_CASE_MULTI(64, 4, 3) SP_ATTN_CASE_MULTI(64, 4, 4)
  // one tile per wave (up to 6 tiles per group; rot can hold only where a
  // compute unit takes two workgroups or more)
  SP_ATTN_CASE(128, 1) SP_ATTN_CASE_ROT(128, 2) SP_ATTN_CASE_ROT(128, 3) SP_ATTN_CASE_ROT(128, 4)
  SP_ATTN_CASE_ROT(128, 5) SP_ATTN_CASE_ROT(128, 6)
  SP_ATTN_CASE(64, 1) SP_ATTN_CASE_ROT(64, 2) SP_ATTN_CASE_ROT(64, 3) SP_ATTN_CASE_ROT(64, 4)
  SP_ATTN_CASE_ROT(64, 5) SP_ATTN_CASE_ROT(64, 6)
#undef SP_ATTN_CASE_MULTI
#undef SP_ATTN_CASE_ROT
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

}  // namespace sp
