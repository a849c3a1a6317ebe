// Host runtime behind the C ABI of include/sp_probe.h: argument checks, split
// planning, workspace layout and the launch sequence of one forward.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <deque>
#include <new>
#include <vector>

#include "../../include/sp_probe.h"
#include "kernels.h"

#include <algorithm>

#define SP_API extern "C" __attribute__((visibility("default")))

namespace {

using namespace sp;

// Profiling: a forward records one event at its start and one after every
// stage (the recursive forward: after every stage of every step), taken from a
// fixed pool used as a ring; the records of the last forwards that still fit
// are kept.
constexpr int kMaxProfiled = 256;
constexpr int kEventPool = kMaxProfiled * (SP_N_STAGES + 1);

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }
int ilog2(int64_t x) { int r = 0; while ((int64_t(1) << r) < x) ++r; return r; }
bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Attention launch shape for `rows` query rows per KV head.
struct AttnPlan {
  int rows, waves, n_qgroups, r_alloc, split_len, max_splits;
};

struct Plan {
  int group, max_tasks, ks, ks_rec, nqkv, esz;
  int q_rows;    // query rows per (sequence, KV head) the one-pass query buffer holds
  AttnPlan rec;  // recursive steps: one soft row (G query rows) per KV head
  // workspace offsets (bytes)
  size_t off_u, off_qkv, off_q, off_ksoft, off_vsoft, off_q_lo, off_ksoft_lo, off_vsoft_lo,
      off_opart, off_ml, off_attn, off_a, off_w, off_s, off_y, off_err;
  // recursive steps only: per-sequence queries and soft keys/values, the fused
  // rows and their inputs
  size_t off_rq, off_rq_lo, off_rks, off_rks_lo, off_rvs, off_rvs_lo, off_rqkv, off_ru, off_rhn,
      off_ren, off_rce, off_rx, off_r3, off_rh0, off_rscale;
  size_t off_gpart, gpart_bytes;  // split-K partial sums of the small-row projections
  size_t total;
};

int check_config(const sp_probe_config* c) {
  if (!c) return SP_ERR_INVALID_ARG;
  if (c->dtype != SP_F32 && c->dtype != SP_BF16) return SP_ERR_INVALID_ARG;
  if (c->pool != SP_POOL_LAST && c->pool != SP_POOL_MEAN) return SP_ERR_INVALID_ARG;
  if (c->hidden <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->intermediate <= 0 ||
      c->k < 1 || c->n_classes < 1 || c->max_batch < 1 || c->max_seq_len < 0)
    return SP_ERR_INVALID_ARG;
  if (c->n_q_heads % c->n_kv_heads) return SP_ERR_INVALID_ARG;
  if (!(c->rms_eps >= 0.0f) || !(c->rope_base > 0.0)) return SP_ERR_INVALID_ARG;
  if (c->split_len != 0 && (c->split_len < 256 || !is_pow2(c->split_len))) return SP_ERR_INVALID_ARG;
  if (c->flags & ~(SP_FLAG_DEBUG | SP_FLAG_PROFILE | SP_FLAG_LAST_ROW_ONLY)) return SP_ERR_INVALID_ARG;
  if ((c->flags & SP_FLAG_LAST_ROW_ONLY) && c->pool != SP_POOL_LAST) return SP_ERR_INVALID_ARG;
  if (c->max_tasks < 0 || c->max_tasks > 64) return SP_ERR_INVALID_ARG;
  if (c->head_dim != 64 && c->head_dim != 128) return SP_ERR_UNSUPPORTED;
  if (c->k > 64 || c->n_classes > 64) return SP_ERR_UNSUPPORTED;
  const int64_t tasks = c->max_tasks > 0 ? c->max_tasks : 1;
  if (tasks * c->k > 1024) return SP_ERR_UNSUPPORTED;
  const int mult = c->dtype == SP_BF16 ? 32 : 4;
  if (c->hidden % mult || c->intermediate % mult) return SP_ERR_UNSUPPORTED;
  if (c->dtype == SP_F32 && tasks * c->k * (c->n_q_heads / c->n_kv_heads) > 64) return SP_ERR_UNSUPPORTED;
  if (c->hidden > 16384) return SP_ERR_UNSUPPORTED;
  if (c->dtype == SP_BF16) {
    // byte offsets inside one MFMA projection operand (activations [B k] rows,
    // or one weight matrix) are 32-bit
    const int64_t qw = (int64_t)c->n_q_heads * c->head_dim;
    const int64_t widest = std::max<int64_t>({c->hidden, qw, c->intermediate});
    const int64_t rows = std::max<int64_t>({(int64_t)c->max_batch * tasks * c->k, qw, c->intermediate});
    if (rows * widest * 2 >= (int64_t(1) << 31)) return SP_ERR_UNSUPPORTED;
  }
  return SP_OK;
}

AttnPlan attn_plan(const sp_probe_config& c, int rows) {
  AttnPlan a{};
  a.rows = rows;
  const int tiles = (rows + 15) / 16;
  if (c.dtype == SP_F32) {
    a.waves = 0;
    a.n_qgroups = 1;
    a.r_alloc = rows;
  } else {
    // one wave per 16-row query tile, at most 12 (head_dim 128: a compute unit
    // holds 12 waves of its ~150 VGPRs) or 16 (64) waves per workgroup, so one
    // workgroup reads each K/V tile for as many rows as fit (the 160 rows of
    // the 27B shape as one group of ten: 28% faster than two groups of five);
    // the sizes below are the instantiated ones (extra tiles are padding)
    static const int kWaves[] = {1, 2, 3, 4, 5, 6, 8, 10, 12, 16};
    const int max_w = c.head_dim == 128 ? 12 : 16;
    const int groups = (tiles + max_w - 1) / max_w;
    const int per_group = (tiles + groups - 1) / groups;
    int w = max_w;
    for (int cand : kWaves)
      if (cand >= per_group) { w = cand; break; }
    a.waves = w;
    a.n_qgroups = (tiles + w - 1) / w;
    a.r_alloc = a.n_qgroups * w * 16;
  }
  if (c.split_len) {
    a.split_len = c.split_len;
  } else if (c.dtype == SP_BF16) {
    // Splits sized so that the attention grid at the full batch and length is
    // at least one round of resident workgroups, and at most a third of the longest
    // sequence: three splits for the longest sequences measured faster than
    // one, two or four on uniform and ragged batches alike, whether the grid
    // is one round or many.  At least 1024 tokens, a multiple of 256.
    const int64_t per_cu = attn_wgs_per_cu(c.head_dim, a.waves);
    const int64_t slots = 256 * std::max<int64_t>(per_cu, 1);
    const int64_t items = (int64_t)c.max_batch * c.n_kv_heads * a.n_qgroups;
    const int64_t want = ((int64_t)c.max_seq_len * items + slots - 1) / slots;
    const int64_t third = ((int64_t)c.max_seq_len + 2) / 3;
    const int64_t sl = (std::min(want, third) + 255) / 256 * 256;
    a.split_len = (int)std::max<int64_t>(sl, 1024);
  } else {
    // fp32 path: at most 8 splits per sequence, between 1024 and 16384 tokens each
    int sl = 1024;
    while (sl < 16384 && (int64_t)sl * 8 < c.max_seq_len) sl *= 2;
    a.split_len = sl;
  }
  a.max_splits = c.max_seq_len > 0 ? (c.max_seq_len + a.split_len - 1) / a.split_len : 1;
  return a;
}

int n_tasks_max(const sp_probe_config& c) { return c.max_tasks > 0 ? c.max_tasks : 1; }

// Attention plan of a one-pass forward with n_tasks tasks: k G query rows per
// task and KV head, or G under SP_FLAG_LAST_ROW_ONLY.
AttnPlan one_pass_plan(const sp_probe_config& c, int n_tasks) {
  const int group = c.n_q_heads / c.n_kv_heads;
  const int per_task = (c.flags & SP_FLAG_LAST_ROW_ONLY) ? 1 : c.k;
  return attn_plan(c, n_tasks * per_task * group);
}

Plan make_plan(const sp_probe_config& c) {
  Plan p{};
  p.esz = c.dtype == SP_BF16 ? 2 : 4;
  p.group = c.n_q_heads / c.n_kv_heads;
  p.max_tasks = n_tasks_max(c);
  p.rec = attn_plan(c, p.group);
  const int S = p.max_tasks * c.k;       // soft rows of the largest call
  p.ks = ((S + 31) / 32) * 32;
  p.ks_rec = ((c.k + 31) / 32) * 32;
  p.nqkv = (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  // split partials: the largest of every plan the handle can run
  size_t part_rows = (size_t)p.rec.max_splits * p.rec.r_alloc;
  p.q_rows = 0;
  for (int t = 1; t <= p.max_tasks; ++t) {
    const AttnPlan a = one_pass_plan(c, t);
    part_rows = std::max(part_rows, (size_t)a.max_splits * a.r_alloc);
    p.q_rows = std::max(p.q_rows, a.r_alloc);
  }

  const size_t B = (size_t)c.max_batch, M = B * S, d = c.hidden, hd = c.head_dim;
  const size_t kv = (size_t)c.n_kv_heads, e = p.esz;
  size_t o = 0;
  auto take = [&](size_t bytes) { const size_t at = o; o = align256(o + bytes); return at; };
  p.off_u = take((size_t)S * d * e);
  p.off_qkv = take((size_t)S * p.nqkv * 4);
  p.off_q = take(B * kv * p.q_rows * hd * e);
  p.off_ksoft = take(B * kv * p.ks * hd * e);
  p.off_vsoft = take(kv * hd * p.ks * e);
  // remainders of the split bf16 queries and soft keys/values (bf16 storage only)
  const size_t lo = c.dtype == SP_BF16 ? 1 : 0;
  p.off_q_lo = take(lo * B * kv * p.q_rows * hd * e);
  p.off_ksoft_lo = take(lo * B * kv * p.ks * hd * e);
  p.off_vsoft_lo = take(lo * kv * hd * p.ks * e);
  p.off_opart = take(B * kv * part_rows * hd * 4);
  p.off_ml = take(B * kv * part_rows * 8);
  p.off_attn = take(M * c.n_q_heads * hd * e);
  p.off_a = take(M * d * 4);
  p.off_w = take(M * d * e);
  p.off_s = take(M * (size_t)c.intermediate * e);
  p.off_y = take(M * d * 4);
  p.off_err = take(256);
  const size_t Mr = B * c.k;
  p.off_rq = take(B * kv * p.rec.r_alloc * hd * e);
  p.off_rq_lo = take(lo * B * kv * p.rec.r_alloc * hd * e);
  p.off_rks = take(B * kv * p.ks_rec * hd * e);
  p.off_rks_lo = take(lo * B * kv * p.ks_rec * hd * e);
  p.off_rvs = take(B * kv * p.ks_rec * hd * e);
  p.off_rvs_lo = take(lo * B * kv * p.ks_rec * hd * e);
  p.off_rqkv = take(B * p.nqkv * 4);
  p.off_ru = take(B * d * e);
  p.off_rhn = take(B * d * e);
  p.off_ren = take((size_t)c.k * d * e);
  p.off_rce = take((size_t)c.k * d * 4);
  p.off_rx = take(Mr * d * 4);
  // Eagle3 input: the three hidden states as scaled fp16 rows, the projected first hidden state
  p.off_r3 = take(B * 3 * d * e);
  p.off_rh0 = take(B * d * 4);
  p.off_rscale = take(B * 4);
  const size_t widest = std::max({(size_t)2 * c.intermediate, (size_t)p.nqkv, d});
  p.gpart_bytes = 16 * 32 * widest * 4;
  p.off_gpart = take(p.gpart_bytes);
  p.total = o;
  return p;
}

}  // namespace

struct sp_probe {
  sp_probe_config cfg;
  Plan plan;
  int device;
  char* ws;
  std::vector<hipEvent_t> events;  // kEventPool events (profiling mode), used as a ring
  struct Record { int start, marks; };
  std::deque<Record> records;      // forwards whose events are still in the pool, oldest first
  int cursor;                      // next free event of the pool
};

namespace {

template <typename T>
T* at(sp_probe* h, size_t off) { return reinterpret_cast<T*>(h->ws + off); }

int check_device() {
  int dev = 0, count = 0;
  if (hipGetDeviceCount(&count) != hipSuccess || count < 1) return SP_ERR_NO_DEVICE;
  if (hipGetDevice(&dev) != hipSuccess) return SP_ERR_NO_DEVICE;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return SP_ERR_NO_DEVICE;
  if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0) return SP_ERR_NO_DEVICE;
  return SP_OK;
}

// Events for a forward of `marks` marks (contiguous in the pool; the oldest
// records they overlap are dropped).  nullptr when profiling is off.
hipEvent_t* prof_begin(sp_probe* h, int marks) {
  if (h->events.empty() || marks > kEventPool) return nullptr;
  if (h->cursor + marks > kEventPool) h->cursor = 0;
  const int lo = h->cursor, hi = h->cursor + marks;
  while (!h->records.empty()) {
    const sp_probe::Record& r = h->records.front();
    if (r.start < hi && r.start + r.marks > lo) h->records.pop_front();
    else break;
  }
  return &h->events[lo];
}

void prof_commit(sp_probe* h, int marks) {
  h->records.push_back({h->cursor, marks});
  h->cursor += marks;
}

// A projection with the handle's split-K scratch.
hipError_t run_gemm(sp_probe* h, DType dt, Epilogue epi, GemmParams g, hipStream_t s) {
  g.part = at<float>(h, h->plan.off_gpart);
  g.part_bytes = h->plan.gpart_bytes;
  return launch_gemm(dt, epi, g, s);
}

// Host-side checks shared by the forwards; *noop is set for an empty batch.
int check_forward(const sp_probe* h, const sp_kv_cache* kv, const int32_t* seq_lens,
                  const int32_t* block_table, const void* soft_prompt, const sp_probe_weights* wt,
                  const float* logits, bool* noop) {
  *noop = false;
  if (!h || !kv || !wt) return SP_ERR_INVALID_ARG;
  const sp_probe_config& c = h->cfg;
  const int B = kv->batch;
  if (B < 0) return SP_ERR_INVALID_ARG;
  if (B > c.max_batch) return SP_ERR_CAPACITY;
  if (B == 0) { *noop = true; return SP_OK; }
  if (!seq_lens || !soft_prompt || !logits) return SP_ERR_INVALID_ARG;
  const void* wptr[11] = {wt->in_norm, wt->w_q, wt->w_k, wt->w_v, wt->w_o, wt->post_norm,
                          wt->w_gate, wt->w_up, wt->w_down, wt->final_norm, wt->w_cls};
  for (const void* q : wptr)
    if (!q || !aligned16(q)) return SP_ERR_INVALID_ARG;
  if (!aligned16(soft_prompt)) return SP_ERR_INVALID_ARG;
  if (wt->cls_rows && (wt->cls_vocab < 1 || ((uintptr_t)wt->cls_rows & 3))) return SP_ERR_INVALID_ARG;
  if (!kv->k_base || !kv->v_base || !aligned16(kv->k_base) || !aligned16(kv->v_base))
    return SP_ERR_INVALID_ARG;
  if (kv->block_size < 16 || !is_pow2(kv->block_size) || kv->max_blocks_per_seq < 1 ||
      kv->num_blocks < 1)
    return SP_ERR_INVALID_ARG;
  const int64_t tile = (int64_t)kv->block_size * c.head_dim;  // elements of one K or V tile
  const int64_t vec = 16 / h->plan.esz;
  if (kv->k_stride_block % vec || kv->k_stride_head % vec || kv->v_stride_block % vec ||
      kv->v_stride_head % vec || kv->k_stride_block < 0 || kv->v_stride_block < 0 ||
      kv->k_stride_head < tile || kv->v_stride_head < tile)
    return SP_ERR_INVALID_ARG;
  if ((int64_t)kv->max_blocks_per_seq * kv->block_size < (int64_t)c.max_seq_len)
    return SP_ERR_INVALID_ARG;  // a sequence of max_seq_len tokens must fit in a table row
  if (!block_table && (int64_t)B * kv->max_blocks_per_seq > kv->num_blocks) return SP_ERR_INVALID_ARG;
  return SP_OK;
}

// Split-attention parameters over the caller's cache for one attention plan.
AttnParams attn_params(const sp_probe_config& c, const AttnPlan& a, const sp_kv_cache* kv,
                       const int32_t* seq_lens, const int32_t* block_table, const int* errp,
                       const void* q, const void* q_lo, float* o_part, float2* ml_part) {
  AttnParams ap{};
  ap.q = q;
  ap.q_lo = q_lo;
  ap.k_base = kv->k_base; ap.v_base = kv->v_base;
  ap.k_sb = kv->k_stride_block; ap.k_sh = kv->k_stride_head;
  ap.v_sb = kv->v_stride_block; ap.v_sh = kv->v_stride_head;
  ap.block_table = block_table;
  ap.seq_lens = seq_lens;
  ap.err = errp;
  ap.o_part = o_part;
  ap.ml_part = ml_part;
  ap.n_kv = c.n_kv_heads; ap.rows = a.rows;
  ap.r_alloc = a.r_alloc; ap.n_qgroups = a.n_qgroups;
  ap.bs_log2 = ilog2(kv->block_size); ap.mbps = kv->max_blocks_per_seq;
  ap.max_seq_len = c.max_seq_len; ap.split_len = a.split_len; ap.max_splits = a.max_splits;
  return ap;
}

GemmParams gemm_one(const void* a, int lda, const void* w, int ldb, void* c, int ldc, int M, int N,
                    int K) {
  GemmParams g{};
  g.a = a;
  g.b[0] = g.b[1] = g.b[2] = w;
  g.b_split0 = g.b_split1 = N;
  g.ldb = ldb;
  g.c = c;
  g.M = M; g.N = N; g.K = K; g.lda = lda; g.ldc = ldc;
  return g;
}

GemmParams gemm_qkv(const sp_probe_config& c, const Plan& pl, const sp_probe_weights* wt,
                    const void* a, void* out, int M) {
  GemmParams g{};
  g.a = a;
  g.b[0] = wt->w_q; g.b[1] = wt->w_k; g.b[2] = wt->w_v;
  g.b_split0 = c.n_q_heads * c.head_dim;
  g.b_split1 = (c.n_q_heads + c.n_kv_heads) * c.head_dim;
  g.ldb = c.hidden;
  g.c = out;
  g.M = M; g.N = pl.nqkv; g.K = c.hidden; g.lda = c.hidden; g.ldc = pl.nqkv;
  return g;
}

GemmParams gemm_gate_up(const sp_probe_config& c, const sp_probe_weights* wt, const void* a,
                        void* out, int M) {
  GemmParams g{};
  g.a = a;
  g.b[0] = wt->w_gate; g.b[1] = wt->w_up; g.b[2] = wt->w_up;
  g.b_split0 = g.b_split1 = 2 * c.intermediate;
  g.ldb = c.hidden;
  g.c = out;
  g.M = M; g.N = 2 * c.intermediate; g.K = c.hidden; g.lda = c.hidden; g.ldc = c.intermediate;
  return g;
}

}  // namespace

SP_API size_t sp_probe_workspace_bytes(const sp_probe_config* cfg) {
  if (check_config(cfg) != SP_OK) return 0;
  return make_plan(*cfg).total;
}

SP_API const char* sp_probe_status_string(int status) {
  switch (status) {
    case SP_OK: return "SP_OK";
    case SP_ERR_INVALID_ARG: return "SP_ERR_INVALID_ARG: invalid argument";
    case SP_ERR_UNSUPPORTED: return "SP_ERR_UNSUPPORTED: configuration not supported";
    case SP_ERR_NO_DEVICE: return "SP_ERR_NO_DEVICE: no gfx950 HIP device";
    case SP_ERR_OUT_OF_MEMORY: return "SP_ERR_OUT_OF_MEMORY: workspace allocation failed";
    case SP_ERR_HIP: return "SP_ERR_HIP: HIP runtime or launch error";
    case SP_ERR_CAPACITY: return "SP_ERR_CAPACITY: batch exceeds max_batch";
    case SP_ERR_DEVICE_DATA: return "SP_ERR_DEVICE_DATA: invalid seq_lens or block ids on the device";
  }
  return "unknown status";
}

SP_API int sp_probe_init(const sp_probe_config* cfg, sp_probe_t** out) {
  if (!out) return SP_ERR_INVALID_ARG;
  *out = nullptr;
  int st = check_config(cfg);
  if (st != SP_OK) return st;
  st = check_device();
  if (st != SP_OK) return st;
  sp_probe* h = new (std::nothrow) sp_probe();
  if (!h) return SP_ERR_OUT_OF_MEMORY;
  h->cfg = *cfg;
  h->plan = make_plan(*cfg);
  h->cursor = 0;
  h->ws = nullptr;
  if (hipGetDevice(&h->device) != hipSuccess) { delete h; return SP_ERR_HIP; }
  if (hipMalloc(&h->ws, h->plan.total) != hipSuccess) { delete h; return SP_ERR_OUT_OF_MEMORY; }
  // Zero once: padded query rows and padded soft key/value slots stay zero for
  // the handle's lifetime (forwards only write the unpadded part).
  if (hipMemset(h->ws, 0, h->plan.total) != hipSuccess || hipDeviceSynchronize() != hipSuccess) {
    (void)hipFree(h->ws);
    delete h;
    return SP_ERR_HIP;
  }
  if (cfg->flags & SP_FLAG_PROFILE) {
    h->events.resize(kEventPool);
    for (auto& ev : h->events) {
      if (hipEventCreate(&ev) != hipSuccess) {
        ev = nullptr;
        sp_probe_destroy(h);
        return SP_ERR_HIP;
      }
    }
  }
  *out = h;
  return SP_OK;
}

SP_API int sp_probe_destroy(sp_probe_t* h) {
  if (!h) return SP_OK;
  int st = SP_OK;
  if (hipDeviceSynchronize() != hipSuccess) st = SP_ERR_HIP;
  for (auto& ev : h->events)
    if (ev) (void)hipEventDestroy(ev);
  if (h->ws && hipFree(h->ws) != hipSuccess) st = SP_ERR_HIP;
  delete h;
  return st;
}

SP_API int sp_probe_plan(const sp_probe_t* h, int32_t batch, int32_t* split_len, int32_t* max_splits,
                         int32_t* rows_per_kv_head, int32_t* query_groups) {
  if (!h || batch < 0) return SP_ERR_INVALID_ARG;
  const AttnPlan a = one_pass_plan(h->cfg, 1);
  if (split_len) *split_len = a.split_len;
  if (max_splits) *max_splits = a.max_splits;
  if (rows_per_kv_head) *rows_per_kv_head = a.rows;
  if (query_groups) *query_groups = a.n_qgroups;
  return SP_OK;
}

SP_API int sp_probe_plan_recursive(const sp_probe_t* h, int32_t batch, int32_t* split_len,
                                   int32_t* max_splits, int32_t* rows_per_kv_head,
                                   int32_t* query_groups) {
  if (!h || batch < 0) return SP_ERR_INVALID_ARG;
  if (split_len) *split_len = h->plan.rec.split_len;
  if (max_splits) *max_splits = h->plan.rec.max_splits;
  if (rows_per_kv_head) *rows_per_kv_head = h->plan.rec.rows;
  if (query_groups) *query_groups = h->plan.rec.n_qgroups;
  return SP_OK;
}

#define SP_TRY(expr) do { if ((expr) != hipSuccess) return SP_ERR_HIP; } while (0)

namespace {

// The one-pass forward for n_tasks tasks (Sec. 3.2-3.3; one task is the plain
// probe): all tasks' soft rows share one pass over the cache.
int forward_one_pass(sp_probe_t* h, const sp_kv_cache* kv, const int32_t* seq_lens,
                     const int32_t* block_table, int n_tasks, const void* soft_prompt,
                     const sp_probe_weights* wt, float* logits, void* stream) {
  // ---- host-side checks: nothing is enqueued unless all pass
  bool noop = false;
  const int chk = check_forward(h, kv, seq_lens, block_table, soft_prompt, wt, logits, &noop);
  if (chk != SP_OK) return chk;
  if (n_tasks < 1 || n_tasks > h->plan.max_tasks) return SP_ERR_INVALID_ARG;
  if (noop) return SP_OK;
  const sp_probe_config& c = h->cfg;
  const Plan& pl = h->plan;
  const int B = kv->batch;

  hipStream_t s = (hipStream_t)stream;
  const DType dt = c.dtype == SP_BF16 ? kBF16 : kF32;   // storage: weights, soft prompt, KV
  const DType at_dt = c.dtype == SP_BF16 ? kF16 : kF32;  // activations feeding the MFMAs
  const int d = c.hidden, hd = c.head_dim, I = c.intermediate, K = c.k;
  const bool last_only = c.flags & SP_FLAG_LAST_ROW_ONLY;
  const int S = n_tasks * K;                 // soft rows (keys and values)
  const int Kq = last_only ? 1 : K;          // rows per task past the attention
  const int R = n_tasks * Kq;                // rows per sequence past the attention
  const int M = B * R;
  const AttnPlan ak = one_pass_plan(c, n_tasks);
  const bool debug = c.flags & SP_FLAG_DEBUG;
  int* err = at<int>(h, pl.off_err);
  const int* errp = debug ? err : nullptr;
  const int marks = SP_N_STAGES + 1;
  hipEvent_t* ev = prof_begin(h, marks);
  int stage = 0;
  auto mark = [&]() -> bool { return !ev || hipEventRecord(ev[stage++], s) == hipSuccess; };

  if (debug) {
    ValidateParams vp{seq_lens, block_table, err, kv->num_blocks, kv->max_blocks_per_seq,
                      ilog2(kv->block_size), c.max_seq_len, wt->cls_rows, n_tasks * c.n_classes, wt->cls_vocab};
    SP_TRY(launch_validate(vp, B, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // stage 0: soft rows — RMSNorm, Q/K/V on the S distinct rows, RoPE per sequence
  SP_TRY(launch_rmsnorm_rows(dt, dt, at_dt, soft_prompt, d, wt->in_norm, nullptr,
                             at<void>(h, pl.off_u), d, S, d, c.rms_eps, s));
  SP_TRY(run_gemm(h, dt, kEpiStore, gemm_qkv(c, pl, wt, at<void>(h, pl.off_u), at<void>(h, pl.off_qkv), S), s));
  {
    RopeParams r{};
    r.qkv = at<float>(h, pl.off_qkv);
    r.seq_lens = seq_lens;
    r.err = errp;
    r.q = at<void>(h, pl.off_q);
    r.k_soft = at<void>(h, pl.off_ksoft);
    r.v_soft = at<void>(h, pl.off_vsoft);
    r.q_lo = at<void>(h, pl.off_q_lo);
    r.k_soft_lo = at<void>(h, pl.off_ksoft_lo);
    r.v_soft_lo = at<void>(h, pl.off_vsoft_lo);
    r.n_q = c.n_q_heads; r.n_kv = c.n_kv_heads; r.hd = hd; r.k = S; r.group = pl.group;
    r.r_alloc = ak.r_alloc; r.ks = pl.ks; r.max_seq_len = c.max_seq_len;
    r.step = 0; r.per_seq = 0;
    r.k_task = K; r.q_first = K - Kq; r.q_per_task = Kq;
    r.rope_base = c.rope_base;
    r.q_scale = (float)(1.4426950408889634 / __builtin_sqrt((double)hd));
    SP_TRY(launch_rope_scatter(dt, r, B, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // stage 1: split attention over the cached K/V
  const AttnParams ap = attn_params(c, ak, kv, seq_lens, block_table, errp, at<void>(h, pl.off_q),
                                    at<void>(h, pl.off_q_lo), at<float>(h, pl.off_opart),
                                    at<float2>(h, pl.off_ml));
  if (dt == kBF16)
    SP_TRY(launch_attention_bf16(ap, hd, ak.waves, B, s));
  else
    SP_TRY(launch_attention_f32(ap, hd, B, s));
  if (!mark()) return SP_ERR_HIP;

  // stage 2: merge the splits and each task's soft keys into the attention output rows
  {
    MergeParams mp{};
    mp.o_part = ap.o_part; mp.ml_part = ap.ml_part; mp.seq_lens = seq_lens; mp.err = errp;
    mp.q = ap.q; mp.q_lo = ap.q_lo;
    mp.k_soft = at<void>(h, pl.off_ksoft); mp.k_soft_lo = at<void>(h, pl.off_ksoft_lo);
    mp.v_soft = at<void>(h, pl.off_vsoft); mp.v_soft_lo = at<void>(h, pl.off_vsoft_lo);
    mp.out = at<void>(h, pl.off_attn);
    mp.n_kv = c.n_kv_heads; mp.group = pl.group; mp.rows = ak.rows;
    mp.r_alloc = ak.r_alloc; mp.hd = hd; mp.ks = pl.ks; mp.max_splits = ak.max_splits;
    mp.split_len = ak.split_len; mp.max_seq_len = c.max_seq_len; mp.n_q = c.n_q_heads;
    mp.k_task = K; mp.q_first = K - Kq; mp.q_per_task = Kq; mp.step = 0;
    mp.out_rows = R; mp.out_off = 0; mp.per_seq = 0;
    SP_TRY(launch_merge(dt, mp, B, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // stage 3: a = x + W_o o, x the row's soft-prompt vector
  {
    const int qw = c.n_q_heads * hd;
    GemmParams g = gemm_one(at<void>(h, pl.off_attn), qw, wt->w_o, qw, at<void>(h, pl.off_a), d, M, d, qw);
    g.r = (const char*)soft_prompt + (size_t)(K - Kq) * d * pl.esz;
    g.r_mod = R;
    g.r_ld = last_only ? K * d : d;
    SP_TRY(run_gemm(h, dt, kEpiResidRow, g, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // stage 4: w = RMSNorm(a; gamma_post)
  SP_TRY(launch_rmsnorm_rows(kF32, dt, at_dt, at<void>(h, pl.off_a), d, wt->post_norm, nullptr,
                             at<void>(h, pl.off_w), d, M, d, c.rms_eps, s));
  if (!mark()) return SP_ERR_HIP;

  // stage 5: s = silu(W_gate w) * (W_up w)
  SP_TRY(run_gemm(h, dt, kEpiSwiglu, gemm_gate_up(c, wt, at<void>(h, pl.off_w), at<void>(h, pl.off_s), M), s));
  if (!mark()) return SP_ERR_HIP;

  // stage 6: y = a + W_down s
  {
    GemmParams g = gemm_one(at<void>(h, pl.off_s), I, wt->w_down, I, at<void>(h, pl.off_y), d, M, d, I);
    g.r = at<void>(h, pl.off_a); g.r_ld = d;
    SP_TRY(run_gemm(h, dt, kEpiResidF32, g, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // stage 7: final RMSNorm, read-out, logits = W_cls pooled (+ b), per task
  {
    ClsParams cp{};
    cp.y = at<float>(h, pl.off_y);
    cp.final_norm = wt->final_norm; cp.w_cls = wt->w_cls; cp.b_cls = wt->b_cls;
    cp.cls_rows = wt->cls_rows; cp.err = errp;
    cp.logits = logits;
    cp.k = Kq; cp.n_tasks = n_tasks; cp.d = d; cp.n_classes = c.n_classes;
    cp.pool_mean = c.pool == SP_POOL_MEAN;
    cp.eps = c.rms_eps;
    SP_TRY(launch_final_classifier(dt, cp, B, s));
  }
  if (!mark()) return SP_ERR_HIP;
  if (ev) prof_commit(h, marks);
  return SP_OK;
}

}  // namespace

SP_API int sp_probe_forward(sp_probe_t* h, const sp_kv_cache* kv, const int32_t* seq_lens,
                            const int32_t* block_table, const void* soft_prompt,
                            const sp_probe_weights* wt, float* logits, void* stream) {
  return forward_one_pass(h, kv, seq_lens, block_table, 1, soft_prompt, wt, logits, stream);
}

SP_API int sp_probe_forward_multi(sp_probe_t* h, const sp_kv_cache* kv, const int32_t* seq_lens,
                                  const int32_t* block_table, int32_t n_tasks, const void* soft_prompts,
                                  const sp_probe_weights* wt, float* logits, void* stream) {
  return forward_one_pass(h, kv, seq_lens, block_table, n_tasks, soft_prompts, wt, logits, stream);
}

SP_API int sp_probe_forward_recursive(sp_probe_t* h, const sp_kv_cache* kv, const int32_t* seq_lens,
                                      const int32_t* block_table, const void* soft_prompt,
                                      const void* hidden_last, const sp_probe_fusion* fusion,
                                      const sp_probe_weights* wt, float* logits, void* stream) {
  // ---- host-side checks: nothing is enqueued unless all pass
  bool noop = false;
  const int chk = check_forward(h, kv, seq_lens, block_table, soft_prompt, wt, logits, &noop);
  if (chk != SP_OK || noop) return chk;
  if (!fusion || !hidden_last || !aligned16(hidden_last)) return SP_ERR_INVALID_ARG;
  const void* fptr[3] = {fusion->fc_norm_hidden, fusion->fc_norm_embed, fusion->w_fc};
  for (const void* q : fptr)
    if (!q || !aligned16(q)) return SP_ERR_INVALID_ARG;
  const bool eagle3 = fusion->w_hidden_fuse != nullptr;
  if (eagle3 && !aligned16(fusion->w_hidden_fuse)) return SP_ERR_INVALID_ARG;
  const sp_probe_config& c = h->cfg;
  const Plan& pl = h->plan;
  const AttnPlan& rp = pl.rec;
  const int B = kv->batch, K = c.k;

  hipStream_t s = (hipStream_t)stream;
  const DType dt = c.dtype == SP_BF16 ? kBF16 : kF32;
  const DType at_dt = c.dtype == SP_BF16 ? kF16 : kF32;
  const int d = c.hidden, hd = c.head_dim, I = c.intermediate, qw = c.n_q_heads * hd;
  const size_t esz = pl.esz;  // bytes of a storage element and of an activation element
  const int64_t ld_steps = (int64_t)K * d;  // row stride of the [B][k][d] step buffers
  const bool debug = c.flags & SP_FLAG_DEBUG;
  int* err = at<int>(h, pl.off_err);
  const int* errp = debug ? err : nullptr;
  const int marks = SP_N_STAGES * K + 1;
  hipEvent_t* ev = prof_begin(h, marks);
  int mk = 0;
  auto mark = [&]() -> bool { return !ev || hipEventRecord(ev[mk++], s) == hipSuccess; };

  char* x_all = at<char>(h, pl.off_rx);   // fused rows x_t: fp32 [B][k][d]
  char* a_all = at<char>(h, pl.off_a);    // a_t: fp32 [B][k][d]
  char* y_all = at<char>(h, pl.off_y);    // y_t: fp32 [B][k][d]
  char* o_all = at<char>(h, pl.off_attn); // attention output: [B][k][n_q hd]
  void* hn = at<void>(h, pl.off_rhn);     // RMSNorm of the hidden state entering a step
  const void* w_fc_embed = (const char*)fusion->w_fc + (size_t)d * esz;  // columns d..2d-1

  if (debug) {
    ValidateParams vp{seq_lens, block_table, err, kv->num_blocks, kv->max_blocks_per_seq,
                      ilog2(kv->block_size), c.max_seq_len, wt->cls_rows, c.n_classes, wt->cls_vocab};
    SP_TRY(launch_validate(vp, B, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // The soft-prompt half of the fusion does not depend on the sequence:
  // c_t = W_fc[:, d:] RMSNorm(e_t; gamma_e) for the k steps, once.
  SP_TRY(launch_rmsnorm_rows(dt, dt, at_dt, soft_prompt, d, fusion->fc_norm_embed, nullptr,
                             at<void>(h, pl.off_ren), d, K, d, c.rms_eps, s));
  SP_TRY(run_gemm(h, dt, kEpiStore, gemm_one(at<void>(h, pl.off_ren), d, w_fc_embed, 2 * d,
                                             at<void>(h, pl.off_rce), d, K, d, d), s));
  if (!eagle3) {
    // the first step's hidden state is the base model's last one
    SP_TRY(launch_rmsnorm_rows(dt, dt, at_dt, hidden_last, d, fusion->fc_norm_hidden, nullptr, hn, d,
                               B, d, c.rms_eps, s));
  } else {
    // Eagle3: the first step's hidden state is W [h_low; h_mid; h_high]; on the
    // bf16 path the three states enter the MFMA as fp16 rows scaled by a power
    // of two (their range can exceed fp16's) and the product is scaled back
    float* h0 = at<float>(h, pl.off_rh0);
    if (dt == kBF16) {
      SP_TRY(launch_scale_rows_f16(hidden_last, 3 * d, at<void>(h, pl.off_r3), at<float>(h, pl.off_rscale),
                                   B, 3 * d, s));
      GemmParams g = gemm_one(at<void>(h, pl.off_r3), 3 * d, fusion->w_hidden_fuse, 3 * d, h0, d, B, d, 3 * d);
      g.r = at<float>(h, pl.off_rscale);
      SP_TRY(run_gemm(h, dt, kEpiRowScale, g, s));
    } else {
      SP_TRY(run_gemm(h, dt, kEpiStore, gemm_one(hidden_last, 3 * d, fusion->w_hidden_fuse, 3 * d, h0, d,
                                                 B, d, 3 * d), s));
    }
    SP_TRY(launch_rmsnorm_rows(kF32, dt, at_dt, h0, d, fusion->fc_norm_hidden, nullptr, hn, d, B, d,
                               c.rms_eps, s));
  }

  for (int t = 0; t < K; ++t) {
    // stage 0: x_t = W_fc[:, :d] RMSNorm(h; gamma_h) + c_t, its RMSNorm, Q/K/V, RoPE at N_b + t
    {
      GemmParams g = gemm_one(hn, d, fusion->w_fc, 2 * d, x_all + (size_t)t * d * 4, (int)ld_steps,
                              B, d, d);
      g.r = at<char>(h, pl.off_rce) + (size_t)t * d * 4; g.r_ld = 0;
      SP_TRY(run_gemm(h, dt, kEpiResidF32, g, s));
    }
    SP_TRY(launch_rmsnorm_rows(kF32, dt, at_dt, x_all + (size_t)t * d * 4, ld_steps, wt->in_norm,
                               nullptr, at<void>(h, pl.off_ru), d, B, d, c.rms_eps, s));
    SP_TRY(run_gemm(h, dt, kEpiStore, gemm_qkv(c, pl, wt, at<void>(h, pl.off_ru), at<void>(h, pl.off_rqkv), B), s));
    {
      RopeParams r{};
      r.qkv = at<float>(h, pl.off_rqkv);
      r.seq_lens = seq_lens;
      r.err = errp;
      r.q = at<void>(h, pl.off_rq);
      r.k_soft = at<void>(h, pl.off_rks);
      r.v_soft = at<void>(h, pl.off_rvs);
      r.q_lo = at<void>(h, pl.off_rq_lo);
      r.k_soft_lo = at<void>(h, pl.off_rks_lo);
      r.v_soft_lo = at<void>(h, pl.off_rvs_lo);
      r.n_q = c.n_q_heads; r.n_kv = c.n_kv_heads; r.hd = hd; r.k = 1; r.group = pl.group;
      r.r_alloc = rp.r_alloc; r.ks = pl.ks_rec; r.max_seq_len = c.max_seq_len;
      r.step = t; r.per_seq = 1;
      r.k_task = 1; r.q_first = 0; r.q_per_task = 1;
      r.rope_base = c.rope_base;
      r.q_scale = (float)(1.4426950408889634 / __builtin_sqrt((double)hd));
      SP_TRY(launch_rope_scatter(dt, r, B, s));
    }
    if (!mark()) return SP_ERR_HIP;

    // stage 1: split attention of the step's G query rows per KV head over the cache
    const AttnParams ap = attn_params(c, rp, kv, seq_lens, block_table, errp, at<void>(h, pl.off_rq),
                                      at<void>(h, pl.off_rq_lo), at<float>(h, pl.off_opart),
                                      at<float2>(h, pl.off_ml));
    if (dt == kBF16)
      SP_TRY(launch_attention_bf16(ap, hd, rp.waves, B, s));
    else
      SP_TRY(launch_attention_f32(ap, hd, B, s));
    if (!mark()) return SP_ERR_HIP;

    // stage 2: merge with the soft keys of steps 0..t into attention rows b*k + t
    {
      MergeParams mp{};
      mp.o_part = ap.o_part; mp.ml_part = ap.ml_part; mp.seq_lens = seq_lens; mp.err = errp;
      mp.q = ap.q; mp.q_lo = ap.q_lo;
      mp.k_soft = at<void>(h, pl.off_rks); mp.k_soft_lo = at<void>(h, pl.off_rks_lo);
      mp.v_soft = at<void>(h, pl.off_rvs); mp.v_soft_lo = at<void>(h, pl.off_rvs_lo);
      mp.out = o_all;
      mp.n_kv = c.n_kv_heads; mp.group = pl.group; mp.rows = rp.rows;
      mp.r_alloc = rp.r_alloc; mp.hd = hd; mp.ks = pl.ks_rec; mp.max_splits = rp.max_splits;
      mp.split_len = rp.split_len; mp.max_seq_len = c.max_seq_len; mp.n_q = c.n_q_heads;
      mp.k_task = 1; mp.q_first = 0; mp.q_per_task = 1; mp.step = t;
      mp.out_rows = K; mp.out_off = t; mp.per_seq = 1;
      SP_TRY(launch_merge(dt, mp, B, s));
    }
    if (!mark()) return SP_ERR_HIP;

    // stage 3: a_t = x_t + W_o o_t
    {
      GemmParams g = gemm_one(o_all + (size_t)t * qw * esz, K * qw, wt->w_o, qw,
                              a_all + (size_t)t * d * 4, (int)ld_steps, B, d, qw);
      g.r = x_all + (size_t)t * d * 4; g.r_ld = (int)ld_steps;
      SP_TRY(run_gemm(h, dt, kEpiResidF32, g, s));
    }
    if (!mark()) return SP_ERR_HIP;

    // stage 4: w = RMSNorm(a_t; gamma_post)
    SP_TRY(launch_rmsnorm_rows(kF32, dt, at_dt, a_all + (size_t)t * d * 4, ld_steps, wt->post_norm,
                               nullptr, at<void>(h, pl.off_w), d, B, d, c.rms_eps, s));
    if (!mark()) return SP_ERR_HIP;

    // stage 5: s = silu(W_gate w) * (W_up w)
    SP_TRY(run_gemm(h, dt, kEpiSwiglu, gemm_gate_up(c, wt, at<void>(h, pl.off_w), at<void>(h, pl.off_s), B), s));
    if (!mark()) return SP_ERR_HIP;

    // stage 6: y_t = a_t + W_down s
    {
      GemmParams g = gemm_one(at<void>(h, pl.off_s), I, wt->w_down, I, y_all + (size_t)t * d * 4,
                              (int)ld_steps, B, d, I);
      g.r = a_all + (size_t)t * d * 4; g.r_ld = (int)ld_steps;
      SP_TRY(run_gemm(h, dt, kEpiResidF32, g, s));
    }
    if (!mark()) return SP_ERR_HIP;

    // stage 7: the step's output f_t = RMSNorm(y_t; gamma_final) is the next
    // step's hidden state, which enters it as RMSNorm(f_t; gamma_h); after the
    // last step, the read-out and the classifier
    if (t + 1 < K) {
      SP_TRY(launch_rmsnorm_rows(kF32, dt, at_dt, y_all + (size_t)t * d * 4, ld_steps, wt->final_norm,
                                 fusion->fc_norm_hidden, hn, d, B, d, c.rms_eps, s));
    } else {
      ClsParams cp{};
      cp.y = (const float*)y_all;
      cp.final_norm = wt->final_norm; cp.w_cls = wt->w_cls; cp.b_cls = wt->b_cls;
      cp.cls_rows = wt->cls_rows; cp.err = errp;
      cp.logits = logits;
      cp.k = K; cp.n_tasks = 1; cp.d = d; cp.n_classes = c.n_classes;
      cp.pool_mean = c.pool == SP_POOL_MEAN;
      cp.eps = c.rms_eps;
      SP_TRY(launch_final_classifier(dt, cp, B, s));
    }
    if (!mark()) return SP_ERR_HIP;
  }
  if (ev) prof_commit(h, marks);
  return SP_OK;
}

#undef SP_TRY

SP_API size_t sp_probe_tap_bytes(const sp_probe_t* h, int tap, int32_t batch) {
  if (!h || batch < 0 || batch > h->cfg.max_batch) return 0;
  const sp_probe_config& c = h->cfg;
  const size_t S = (size_t)h->plan.max_tasks * c.k, M = (size_t)batch * S, e = h->plan.esz;
  switch (tap) {
    case SP_TAP_QKV: return S * h->plan.nqkv * 4;
    case SP_TAP_ATTN: return M * c.n_q_heads * c.head_dim * e;
    case SP_TAP_A: return M * c.hidden * 4;
    case SP_TAP_Y: return M * c.hidden * 4;
    case SP_TAP_X: return (size_t)batch * c.k * c.hidden * 4;
  }
  return 0;
}

SP_API int sp_probe_copy_tap(sp_probe_t* h, int tap, int32_t batch, void* dst, size_t dst_bytes,
                             void* stream) {
  const size_t n = sp_probe_tap_bytes(h, tap, batch);
  if (!h || !dst || n == 0 || dst_bytes < n) return SP_ERR_INVALID_ARG;
  size_t off = 0;
  switch (tap) {
    case SP_TAP_QKV: off = h->plan.off_qkv; break;
    case SP_TAP_ATTN: off = h->plan.off_attn; break;
    case SP_TAP_A: off = h->plan.off_a; break;
    case SP_TAP_Y: off = h->plan.off_y; break;
    case SP_TAP_X: off = h->plan.off_rx; break;
  }
  if (hipMemcpyAsync(dst, h->ws + off, n, hipMemcpyDeviceToDevice, (hipStream_t)stream) != hipSuccess)
    return SP_ERR_HIP;
  return SP_OK;
}

SP_API int sp_probe_check_device_error(sp_probe_t* h, void* stream) {
  if (!h) return SP_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  int val = 0;
  if (hipStreamSynchronize(s) != hipSuccess) return SP_ERR_HIP;
  if (hipMemcpy(&val, h->ws + h->plan.off_err, sizeof(int), hipMemcpyDeviceToHost) != hipSuccess)
    return SP_ERR_HIP;
  if (val) {
    if (hipMemset(h->ws + h->plan.off_err, 0, sizeof(int)) != hipSuccess ||
        hipDeviceSynchronize() != hipSuccess)
      return SP_ERR_HIP;
    return SP_ERR_DEVICE_DATA;
  }
  return SP_OK;
}

SP_API int sp_probe_profile_read(sp_probe_t* h, float* stage_ms, int32_t n_stages, int32_t* n_forwards) {
  if (!h || !stage_ms || n_stages < 1 || n_stages > SP_N_STAGES) return SP_ERR_INVALID_ARG;
  if (!(h->cfg.flags & SP_FLAG_PROFILE)) return SP_ERR_INVALID_ARG;
  for (int i = 0; i < n_stages; ++i) stage_ms[i] = 0.f;
  for (const sp_probe::Record& r : h->records) {
    hipEvent_t* ev = &h->events[r.start];
    if (hipEventSynchronize(ev[r.marks - 1]) != hipSuccess) return SP_ERR_HIP;
    for (int i = 0; i + 1 < r.marks; ++i) {
      const int st = i % SP_N_STAGES;
      if (st >= n_stages) continue;
      float ms = 0.f;
      if (hipEventElapsedTime(&ms, ev[i], ev[i + 1]) != hipSuccess) return SP_ERR_HIP;
      stage_ms[st] += ms;
    }
  }
  if (n_forwards) *n_forwards = (int32_t)h->records.size();
  h->records.clear();
  h->cursor = 0;
  return SP_OK;
}
