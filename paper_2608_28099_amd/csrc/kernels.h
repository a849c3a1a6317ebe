// Internal interface between the host runtime and the kernels (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sp {

// Storage types; bf16-storage configs compute with fp16 activations (kF16).
enum DType { kF32 = 0, kBF16 = 1, kF16 = 2 };

// Bits of the status word a forward's kernels set (atomic OR) on conditions the
// host cannot see: a seq_len outside [0, max_seq_len] (the kernels clamp it),
// and an fp16 activation that left fp16's range (stored as inf).
enum StatusBits { kStatusSeqLen = 16, kStatusRange = 32 };

// ---------------------------------------------------------------- soft-row prep
// out[r][i] = x[r][i] / sqrt(mean_i x[r][i]^2 + eps) * gain[i], rows r < rows
// (row strides ld_x, ld_out in elements).  gain2 (nullable): the result is
// normed once more with gain2 (RMSNorm(RMSNorm(x; gain); gain2)), in fp32.
// status (nullable): kStatusRange is set if an fp16 output exceeds fp16's range.
hipError_t launch_rmsnorm_rows(DType in_dt, DType gain_dt, DType out_dt, const void* x,
                               int64_t ld_x, const void* gain, const void* gain2, void* out,
                               int64_t ld_out, int rows, int d, float eps, int* status,
                               hipStream_t s);

// Soft rows j = 0..k-1 of a launch belong to tasks of k_task rows each (one-pass:
// every task's soft prompt; recursive: k = k_task = 1).  Row j of its task
// (jj = j % k_task) sits at position N_b + step + jj and fills soft key/value
// slot step + j; only rows jj >= q_first carry queries, which go to query row
// (j / k_task) * q_per_task + jj - q_first of the sequence.
struct RopeParams {
  const float* qkv;        // [k][(n_q + 2 n_kv) hd] fp32 ([B][k][...] when per_seq)
  const int* seq_lens;     // device [B]
  const int* err;          // nullable: skip everything if *err != 0
  int* status;             // kStatusSeqLen for a seq_len outside [0, max_seq_len]
  void* q;                 // [B][n_kv][r_alloc][hd], scaled by q_scale
  void* k_soft;            // [B][n_kv][ks][hd] (rotated soft keys)
  void* v_soft;            // [n_kv][ks][hd] (batch-invariant), or [B][n_kv][ks][hd] (per_seq)
  // bf16 split output (dt == kBF16): q, k_soft, v_soft receive bf16(x) and these
  // the remainders bf16(x - bf16(x)), same layouts
  void* q_lo;
  void* k_soft_lo;
  void* v_soft_lo;
  int n_q, n_kv, hd, k, group, r_alloc, ks, max_seq_len;
  int step;                // position and slot offset (recursive step)
  int per_seq;             // projections and values per sequence (recursive steps)
  int k_task, q_first, q_per_task;
  double rope_base;
  float q_scale;           // log2(e) / sqrt(hd)
  int num_cus;             // compute units of the device (sizes the grid)
};
// dt: output type: kF32, or kBF16 for the hi/lo bf16 split
hipError_t launch_rope_scatter(DType dt, const RopeParams& p, int batch, hipStream_t s);

// fp16 copy of bf16 rows scaled by a power of two so that no value exceeds the
// fp16 range: out[r][i] = x[r][i] * 2^-e_r, inv_scale[r] = 2^e_r, with e_r >= 0
// the smallest exponent that brings max_i |x[r][i]| * 2^-e_r below 2^15.
hipError_t launch_scale_rows_f16(const void* x, int64_t ld_x, void* out, float* inv_scale, int rows,
                                 int cols, hipStream_t s);

// ---------------------------------------------------------------- attention
struct AttnParams {
  const void* q;           // [B][n_kv][r_alloc][hd], pre-scaled by log2(e)/sqrt(hd)
  const void* q_lo;        // bf16 path: remainders of q (same layout)
  const void* k_base;
  const void* v_base;
  int64_t k_sb, k_sh, v_sb, v_sh;     // elements
  const int* block_table;  // nullable (contiguous)
  const int* seq_lens;
  // nullable (bf16 path: from launch_work_list): the (sequence, split) of grid
  // slot y + max_splits z, for the first *n_items slots; later slots exit
  const int2* items;
  const int* n_items;
  const int* err;          // nullable
  // [B][n_kv][max_splits][r_alloc][hd]: bf16 path fp16 O / l (each split's
  // output normalised by its own sum; 0 for a split with no tokens), fp32 path
  // fp32 unnormalised O
  void* o_part;
  float2* ml_part;         // [B][n_kv][max_splits][r_alloc] (running max (log2 units), sum)
  int n_kv, rows, r_alloc, n_qgroups;
  int n_tiles;             // 16-row query tiles per query group (r_alloc = n_qgroups n_tiles 16)
  int bs_log2, mbps, max_seq_len, split_len, max_splits;
  int num_cus;             // compute units of the device
  int f16;                 // bf16 path: single fp16 products (K, V converted in LDS; Q, P in fp16)
  int stages;              // bf16 path: LDS stages of the load pipeline (3)
};
// Workgroups of the bf16 attention kernel one compute unit holds: by LDS (160 KB;
// three stages, each a 32-token unit of K and V: 16.4 KB at head_dim 128) and by
// VGPRs: one query tile per wave takes ~150 (12 waves per compute unit at
// head_dim 128, 20 at 64), several tiles per wave ~250 (8 waves).
inline int attn_wgs_per_cu(int hd, int waves, int tiles_per_wave = 1) {
  const int stage_bytes = (hd == 128 ? 1028 : 516) * 16;
  const int by_lds = (160 * 1024) / (3 * stage_bytes + 4096);
  const int by_vgprs = (tiles_per_wave > 1 ? 8 : (hd == 128 ? 12 : 20)) / waves;
  return by_vgprs < by_lds ? by_vgprs : by_lds;
}
// Cache tokens only (the soft keys are folded in by the merge).
// bf16-storage path (bf16 MFMA, split Q and P): head_dim 64/128, `waves` 16-row
// query tiles per workgroup (1, 2, 3, 4, 5, 6, 8, 10 or 12; up to 16 for head_dim 64).
hipError_t launch_attention_bf16(const AttnParams& p, int hd, int waves, int batch, hipStream_t s);
// fp32 VALU path: head_dim 64/128, rows <= 64.
hipError_t launch_attention_f32(const AttnParams& p, int hd, int batch, hipStream_t s);
// The split attention's work items in dispatch order (longest first): every
// split that is not its sequence's last (split_len tokens each), by sequence
// and split; then each sequence's last split (split 0 of an empty sequence),
// by token count descending, ties by sequence.  items holds batch * max_splits
// pairs (sequence, split); *count receives the number written.
hipError_t launch_work_list(const int* seq_lens, int batch, int max_seq_len, int split_len, int2* items, int* count,
                            hipStream_t s);

struct MergeParams {
  const void* o_part;      // as AttnParams::o_part
  const float2* ml_part;
  const int* seq_lens;
  const int* err;
  // the soft keys, in the layouts rope_scatter writes (bf16 path: hi and lo parts)
  const void* q;
  const void* q_lo;
  const void* k_soft;
  const void* k_soft_lo;
  const void* v_soft;
  const void* v_soft_lo;
  void* out;               // [B out_rows][n_q hd] (activation dtype)
  int* status;             // kStatusRange if an fp16 output exceeds fp16's range
  int min_wgs;             // fewest workgroups the soft-row blocking may leave (4 per compute unit)
  int n_kv, group, rows, r_alloc, hd, ks, max_splits, split_len, max_seq_len, n_q;
  // Row r holds query qi = r / group of its sequence: soft row
  // j = (qi / q_per_task) * k_task + q_first + qi % q_per_task + step, which
  // sees the soft keys of its own task up to itself, [(qi / q_per_task) * k_task, j];
  // its output goes to row b * out_rows + out_off + qi.
  int k_task, q_first, q_per_task, step, out_rows, out_off;
  int per_seq;             // v_soft is [B][n_kv][ks][hd] instead of [n_kv][ks][hd]
  int rw;                  // soft rows per workgroup (set by launch_merge)
};
// dt: storage dtype of the config (the output is fp16 for bf16 storage)
hipError_t launch_merge(DType dt, const MergeParams& p, int batch, hipStream_t s);

// ---------------------------------------------------------------- GEMM
enum Epilogue {
  kEpiStore = 0,      // C fp32 = acc
  kEpiResidRow = 1,   // C fp32 = acc + R[(m % r_mod) * r_ld + n]   (R in the storage dtype)
  kEpiResidF32 = 2,   // C fp32 = acc + R[m * r_ld + n]   (R fp32; r_ld 0 = one row for all m)
  kEpiSwiglu = 3,     // C (activation dtype) [m][n] = silu(acc_gate) * acc_up, n < N/2
  kEpiRowScale = 4    // C fp32 = acc * R[m]               (R fp32, one factor per row)
};
struct GemmParams {
  const void* a;           // [M][lda], activation dtype (fp16 for bf16 storage)
  const void* b[3];        // weight row blocks: rows [0, b_split0) from b[0], [b_split0, b_split1)
                           // from b[1], the rest from b[2]; SwiGLU: b[0] gate, b[1] up
  int b_split0, b_split1;
  int ldb;                 // row stride of every b[i]
  void* c;
  const void* r;           // residual
  int M, N, K, lda, ldc, r_mod, r_ld;
  // nullable scratch for split-K partial sums of small-M products (fp32); the
  // launcher splits K only when the partials fit in part_bytes
  float* part;
  size_t part_bytes;
  int* status;             // kStatusRange if an fp16 SwiGLU output exceeds fp16's range
  int b_f16;               // the weight blocks are fp16 (a converted image), not bf16
  int n_cus, n_xcd;        // compute units and XCDs of the device
  int group_m;             // row tiles per group of the tile order (0: the launcher's choice)
};
// dt: storage dtype of the weights (kF32: fp32 VALU path; kBF16: fp16 MFMA path)
hipError_t launch_gemm(DType dt, Epilogue epi, const GemmParams& p, hipStream_t s);
// One tile shape of the fp16 MFMA path (index into the tile table of gemm.hip),
// K split ksplit ways: for measurement; launch_gemm chooses for the forward.
hipError_t launch_gemm_tile(Epilogue epi, const GemmParams& p, int tile, int ksplit, hipStream_t s);
// Sum of ksplit fp32 partial slices in p.part and the epilogue (tile width bn,
// for the SwiGLU column interleave).
hipError_t launch_gemm_reduce(Epilogue epi, const GemmParams& p, int ksplit, int bn, hipStream_t s);

// ---------------------------------------------------------------- read-out
struct ClsParams {
  const float* y;          // [B][n_tasks][k][d]: k rows per task
  const void* final_norm;  // [d]
  const void* w_cls;       // [n_tasks][C][d]
  const float* b_cls;      // nullable, [n_tasks][C]
  const int* cls_rows;     // nullable, [n_tasks][C]: row of w_cls (a vocabulary matrix) per class
  const int* err;          // nullable: skip everything if *err != 0
  float* logits;           // [B][n_tasks][C]
  int k, d, n_classes, pool_mean, n_tasks;
  float eps;
};
hipError_t launch_final_classifier(DType dt, const ClsParams& p, int batch, hipStream_t s);

// ---------------------------------------------------------------- debug validation
struct ValidateParams {
  const int* seq_lens;
  const int* block_table;  // nullable
  int* err;
  int64_t num_blocks;
  int mbps, bs_log2, max_seq_len;
  const int* cls_rows;     // nullable: n_cls_rows row indices, each < cls_vocab
  int n_cls_rows;
  int64_t cls_vocab;
};
hipError_t launch_validate(const ValidateParams& p, int batch, hipStream_t s);

// ---------------------------------------------------------------- workspace guards, weight image
// Fill n 32-bit words at p with `value` (a kernel, so it may be captured in a graph).
hipError_t launch_fill_words(uint32_t* p, size_t n, uint32_t value, hipStream_t s);
// Check n_guards guard areas of `words` 32-bit words each, at byte offsets
// offs[i] (device array) from base, against `value`; *flag |= bit on a mismatch.
hipError_t launch_check_guards(const char* base, const uint64_t* offs, int n_guards, int words,
                               uint32_t value, int* flag, int bit, hipStream_t s);
// fp16 copy of n bf16 values (exact for magnitudes in fp16's normal range; the
// same conversion the projections apply to bf16 weights per fragment).
hipError_t launch_bf16_to_f16(const void* src, void* dst, size_t n, hipStream_t s);
// Compare the n_words header words at image against expect (device); *flag |= bit on a mismatch.
hipError_t launch_check_header(const uint32_t* image, const uint32_t* expect, int n_words, int* flag,
                               int bit, hipStream_t s);

}  // namespace sp
