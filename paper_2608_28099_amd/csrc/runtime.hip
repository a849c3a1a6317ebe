// Host runtime behind the C ABI of include/sp_probe.h: argument checks, split
// planning, workspace layout and the launch sequence of one forward.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <new>
#include <vector>

#include "../../include/sp_probe.h"
#include "kernels.h"

#include <algorithm>

#define SP_API extern "C" __attribute__((visibility("default")))

namespace {

using namespace sp;

constexpr int kMaxProfiled = 256;
constexpr int kEventsPerForward = SP_N_STAGES + 1;

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }
int ilog2(int64_t x) { int r = 0; while ((int64_t(1) << r) < x) ++r; return r; }
bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

struct Plan {
  int group, rows, waves, n_qgroups, r_alloc, ks, nqkv, split_len, max_splits, esz;
  // workspace offsets (bytes)
  size_t off_u, off_qkv, off_q, off_ksoft, off_vsoft, off_q_lo, off_ksoft_lo, off_vsoft_lo,
      off_opart, off_ml, off_attn, off_a, off_w, off_s, off_y, off_err, total;
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
  if (c->flags & ~(SP_FLAG_DEBUG | SP_FLAG_PROFILE)) return SP_ERR_INVALID_ARG;
  if (c->head_dim != 64 && c->head_dim != 128) return SP_ERR_UNSUPPORTED;
  if (c->k > 64 || c->n_classes > 64) return SP_ERR_UNSUPPORTED;
  const int mult = c->dtype == SP_BF16 ? 32 : 4;
  if (c->hidden % mult || c->intermediate % mult) return SP_ERR_UNSUPPORTED;
  if (c->dtype == SP_F32 && c->k * (c->n_q_heads / c->n_kv_heads) > 64) return SP_ERR_UNSUPPORTED;
  if (c->hidden > 16384) return SP_ERR_UNSUPPORTED;
  return SP_OK;
}

Plan make_plan(const sp_probe_config& c) {
  Plan p{};
  p.esz = c.dtype == SP_BF16 ? 2 : 4;
  p.group = c.n_q_heads / c.n_kv_heads;
  p.rows = c.k * p.group;
  const int tiles = (p.rows + 15) / 16;
  if (c.dtype == SP_F32) {
    p.waves = 0;
    p.n_qgroups = 1;
    p.r_alloc = p.rows;
  } else {
    // one wave per 16-row query tile, at most 8 (head_dim 128) or 16 (64) waves
    // per workgroup, whose register budget then still fits without spills; the
    // sizes below are the instantiated ones (extra tiles are padding)
    static const int kWaves[] = {1, 2, 3, 4, 5, 6, 8, 10, 12, 16};
    const int max_w = c.head_dim == 128 ? 8 : 16;
    const int groups = (tiles + max_w - 1) / max_w;
    const int per_group = (tiles + groups - 1) / groups;
    int w = max_w;
    for (int cand : kWaves)
      if (cand >= per_group) { w = cand; break; }
    p.waves = w;
    p.n_qgroups = (tiles + w - 1) / w;
    p.r_alloc = p.n_qgroups * w * 16;
  }
  p.ks = ((c.k + 31) / 32) * 32;
  p.nqkv = (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  if (c.split_len) {
    p.split_len = c.split_len;
  } else if (c.dtype == SP_BF16) {
    // Splits sized so that the attention grid at the full batch and length is
    // about one round of resident workgroups (256 compute units x 3 workgroups
    // of <= 4 waves, x 2 above): every round of workgroups costs a start-up
    // and a drain.  At most max_seq_len / 2 (two splits for the longest
    // sequence, so batches of mixed lengths still balance), at least 1024,
    // a multiple of 256.
    const int64_t slots = 256 * (p.waves <= 4 ? 3 : 2);
    const int64_t items = (int64_t)c.max_batch * c.n_kv_heads * p.n_qgroups;
    const int64_t want = ((int64_t)c.max_seq_len * items + slots - 1) / slots;
    const int64_t half = ((int64_t)c.max_seq_len / 2 + 255) / 256 * 256;
    int64_t sl = (want + 255) / 256 * 256;
    sl = std::min(sl, half);
    p.split_len = (int)std::max<int64_t>(sl, 1024);
  } else {
    // fp32 path: at most 8 splits per sequence, between 1024 and 16384 tokens each
    int sl = 1024;
    while (sl < 16384 && (int64_t)sl * 8 < c.max_seq_len) sl *= 2;
    p.split_len = sl;
  }
  p.max_splits = c.max_seq_len > 0 ? (c.max_seq_len + p.split_len - 1) / p.split_len : 1;

  const size_t B = (size_t)c.max_batch, M = B * c.k, d = c.hidden, hd = c.head_dim;
  const size_t e = p.esz;
  size_t o = 0;
  auto take = [&](size_t bytes) { const size_t at = o; o = align256(o + bytes); return at; };
  p.off_u = take((size_t)c.k * d * e);
  p.off_qkv = take((size_t)c.k * p.nqkv * 4);
  p.off_q = take(B * c.n_kv_heads * p.r_alloc * hd * e);
  p.off_ksoft = take(B * c.n_kv_heads * p.ks * hd * e);
  p.off_vsoft = take((size_t)c.n_kv_heads * hd * p.ks * e);
  // remainders of the split bf16 queries and soft keys/values (bf16 storage only)
  const size_t lo = c.dtype == SP_BF16 ? 1 : 0;
  p.off_q_lo = take(lo * B * c.n_kv_heads * p.r_alloc * hd * e);
  p.off_ksoft_lo = take(lo * B * c.n_kv_heads * p.ks * hd * e);
  p.off_vsoft_lo = take(lo * (size_t)c.n_kv_heads * hd * p.ks * e);
  p.off_opart = take(B * c.n_kv_heads * p.max_splits * p.r_alloc * hd * 4);
  p.off_ml = take(B * c.n_kv_heads * p.max_splits * p.r_alloc * 8);
  p.off_attn = take(M * c.n_q_heads * hd * e);
  p.off_a = take(M * d * 4);
  p.off_w = take(M * d * e);
  p.off_s = take(M * (size_t)c.intermediate * e);
  p.off_y = take(M * d * 4);
  p.off_err = take(256);
  p.total = o;
  return p;
}

}  // namespace

struct sp_probe {
  sp_probe_config cfg;
  Plan plan;
  int device;
  char* ws;
  std::vector<hipEvent_t> events;  // kMaxProfiled * kEventsPerForward, used as a ring
  int64_t n_profiled;
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
  h->n_profiled = 0;
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
    h->events.resize((size_t)kMaxProfiled * kEventsPerForward);
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
  if (split_len) *split_len = h->plan.split_len;
  if (max_splits) *max_splits = h->plan.max_splits;
  if (rows_per_kv_head) *rows_per_kv_head = h->plan.rows;
  if (query_groups) *query_groups = h->plan.n_qgroups;
  return SP_OK;
}

SP_API int sp_probe_forward(sp_probe_t* h, const sp_kv_cache* kv, const int32_t* seq_lens,
                            const int32_t* block_table, const void* soft_prompt,
                            const sp_probe_weights* wt, float* logits, void* stream) {
  // ---- host-side checks: nothing is enqueued unless all pass
  if (!h || !kv || !wt) return SP_ERR_INVALID_ARG;
  const sp_probe_config& c = h->cfg;
  const Plan& pl = h->plan;
  const int B = kv->batch;
  if (B < 0) return SP_ERR_INVALID_ARG;
  if (B > c.max_batch) return SP_ERR_CAPACITY;
  if (B == 0) return SP_OK;
  if (!seq_lens || !soft_prompt || !logits) return SP_ERR_INVALID_ARG;
  const void* wptr[11] = {wt->in_norm, wt->w_q, wt->w_k, wt->w_v, wt->w_o, wt->post_norm,
                          wt->w_gate, wt->w_up, wt->w_down, wt->final_norm, wt->w_cls};
  for (const void* q : wptr)
    if (!q || !aligned16(q)) return SP_ERR_INVALID_ARG;
  if (!aligned16(soft_prompt)) return SP_ERR_INVALID_ARG;
  if (!kv->k_base || !kv->v_base || !aligned16(kv->k_base) || !aligned16(kv->v_base))
    return SP_ERR_INVALID_ARG;
  if (kv->block_size < 16 || !is_pow2(kv->block_size) || kv->max_blocks_per_seq < 1 ||
      kv->num_blocks < 1)
    return SP_ERR_INVALID_ARG;
  const int64_t tile = (int64_t)kv->block_size * c.head_dim;  // elements of one K or V tile
  const int64_t vec = 16 / pl.esz;
  if (kv->k_stride_block % vec || kv->k_stride_head % vec || kv->v_stride_block % vec ||
      kv->v_stride_head % vec || kv->k_stride_block < 0 || kv->v_stride_block < 0 ||
      kv->k_stride_head < tile || kv->v_stride_head < tile)
    return SP_ERR_INVALID_ARG;
  if ((int64_t)kv->max_blocks_per_seq * kv->block_size < (int64_t)c.max_seq_len)
    return SP_ERR_INVALID_ARG;  // a sequence of max_seq_len tokens must fit in a table row
  if (!block_table && (int64_t)B * kv->max_blocks_per_seq > kv->num_blocks) return SP_ERR_INVALID_ARG;

  hipStream_t s = (hipStream_t)stream;
  const DType dt = c.dtype == SP_BF16 ? kBF16 : kF32;   // storage: weights, soft prompt, KV
  const DType at_dt = c.dtype == SP_BF16 ? kF16 : kF32;  // activations feeding the MFMAs
  const int d = c.hidden, hd = c.head_dim, I = c.intermediate, M = B * c.k;
  const bool debug = c.flags & SP_FLAG_DEBUG;
  const bool prof = c.flags & SP_FLAG_PROFILE;
  int* err = at<int>(h, pl.off_err);
  const int* errp = debug ? err : nullptr;
  hipEvent_t* ev = nullptr;
  if (prof) ev = &h->events[(size_t)(h->n_profiled % kMaxProfiled) * kEventsPerForward];
  int stage = 0;
  auto mark = [&]() -> bool { return !prof || hipEventRecord(ev[stage++], s) == hipSuccess; };
#define SP_TRY(expr) do { if ((expr) != hipSuccess) return SP_ERR_HIP; } while (0)

  if (debug) {
    ValidateParams vp{seq_lens, block_table, err, kv->num_blocks, kv->max_blocks_per_seq,
                      ilog2(kv->block_size), c.max_seq_len};
    SP_TRY(launch_validate(vp, B, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // stage 0: soft rows — RMSNorm, Q/K/V on the k distinct rows, RoPE per sequence
  SP_TRY(launch_rmsnorm_rows(dt, dt, at_dt, soft_prompt, wt->in_norm, at<void>(h, pl.off_u), c.k, d,
                             c.rms_eps, s));
  {
    GemmParams g{};
    g.a = at<void>(h, pl.off_u);
    g.b[0] = wt->w_q; g.b[1] = wt->w_k; g.b[2] = wt->w_v;
    g.b_split0 = c.n_q_heads * hd;
    g.b_split1 = (c.n_q_heads + c.n_kv_heads) * hd;
    g.ldb = d;
    g.c = at<void>(h, pl.off_qkv);
    g.M = c.k; g.N = pl.nqkv; g.K = d; g.lda = d; g.ldc = pl.nqkv;
    SP_TRY(launch_gemm(dt, kEpiStore, g, s));
  }
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
    r.n_q = c.n_q_heads; r.n_kv = c.n_kv_heads; r.hd = hd; r.k = c.k; r.group = pl.group;
    r.r_alloc = pl.r_alloc; r.ks = pl.ks; r.max_seq_len = c.max_seq_len;
    r.rope_base = c.rope_base;
    r.q_scale = (float)(1.4426950408889634 / __builtin_sqrt((double)hd));
    SP_TRY(launch_rope_scatter(dt, r, B, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // stage 1: split attention over [cached K/V ; soft K/V]
  AttnParams ap{};
  ap.q = at<void>(h, pl.off_q);
  ap.q_lo = at<void>(h, pl.off_q_lo);
  ap.k_base = kv->k_base; ap.v_base = kv->v_base;
  ap.k_sb = kv->k_stride_block; ap.k_sh = kv->k_stride_head;
  ap.v_sb = kv->v_stride_block; ap.v_sh = kv->v_stride_head;
  ap.block_table = block_table;
  ap.seq_lens = seq_lens;
  ap.err = errp;
  ap.o_part = at<float>(h, pl.off_opart);
  ap.ml_part = at<float2>(h, pl.off_ml);
  ap.n_kv = c.n_kv_heads; ap.rows = pl.rows;
  ap.r_alloc = pl.r_alloc; ap.n_qgroups = pl.n_qgroups;
  ap.bs_log2 = ilog2(kv->block_size); ap.mbps = kv->max_blocks_per_seq;
  ap.max_seq_len = c.max_seq_len; ap.split_len = pl.split_len; ap.max_splits = pl.max_splits;
  if (dt == kBF16)
    SP_TRY(launch_attention_bf16(ap, hd, pl.waves, B, s));
  else
    SP_TRY(launch_attention_f32(ap, hd, B, s));
  if (!mark()) return SP_ERR_HIP;

  // stage 2: merge the splits into the attention output rows b*k + j
  {
    MergeParams mp{};
    mp.o_part = ap.o_part; mp.ml_part = ap.ml_part; mp.seq_lens = seq_lens; mp.err = errp;
    mp.q = ap.q; mp.q_lo = ap.q_lo;
    mp.k_soft = at<void>(h, pl.off_ksoft); mp.k_soft_lo = at<void>(h, pl.off_ksoft_lo);
    mp.v_soft = at<void>(h, pl.off_vsoft); mp.v_soft_lo = at<void>(h, pl.off_vsoft_lo);
    mp.out = at<void>(h, pl.off_attn);
    mp.n_kv = c.n_kv_heads; mp.group = pl.group; mp.k = c.k; mp.rows = pl.rows;
    mp.r_alloc = pl.r_alloc; mp.hd = hd; mp.ks = pl.ks; mp.max_splits = pl.max_splits;
    mp.split_len = pl.split_len; mp.max_seq_len = c.max_seq_len; mp.n_q = c.n_q_heads;
    SP_TRY(launch_merge(dt, mp, B, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // stage 3: a = x_j + W_o o
  {
    GemmParams g{};
    g.a = at<void>(h, pl.off_attn);
    g.b[0] = g.b[1] = g.b[2] = wt->w_o;
    g.b_split0 = g.b_split1 = d;
    g.ldb = c.n_q_heads * hd;
    g.c = at<void>(h, pl.off_a);
    g.r = soft_prompt; g.r_mod = c.k;
    g.M = M; g.N = d; g.K = c.n_q_heads * hd; g.lda = c.n_q_heads * hd; g.ldc = d;
    SP_TRY(launch_gemm(dt, kEpiResidRow, g, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // stage 4: w = RMSNorm(a; gamma_post)
  SP_TRY(launch_rmsnorm_rows(kF32, dt, at_dt, at<void>(h, pl.off_a), wt->post_norm,
                             at<void>(h, pl.off_w), M, d, c.rms_eps, s));
  if (!mark()) return SP_ERR_HIP;

  // stage 5: s = silu(W_gate w) * (W_up w)
  {
    GemmParams g{};
    g.a = at<void>(h, pl.off_w);
    g.b[0] = wt->w_gate; g.b[1] = wt->w_up; g.b[2] = wt->w_up;
    g.b_split0 = g.b_split1 = 2 * I;
    g.ldb = d;
    g.c = at<void>(h, pl.off_s);
    g.M = M; g.N = 2 * I; g.K = d; g.lda = d; g.ldc = I;
    SP_TRY(launch_gemm(dt, kEpiSwiglu, g, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // stage 6: y = a + W_down s
  {
    GemmParams g{};
    g.a = at<void>(h, pl.off_s);
    g.b[0] = g.b[1] = g.b[2] = wt->w_down;
    g.b_split0 = g.b_split1 = d;
    g.ldb = I;
    g.c = at<void>(h, pl.off_y);
    g.r = at<void>(h, pl.off_a);
    g.M = M; g.N = d; g.K = I; g.lda = I; g.ldc = d;
    SP_TRY(launch_gemm(dt, kEpiResidF32, g, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // stage 7: final RMSNorm, read-out, logits = W_cls pooled (+ b)
  {
    ClsParams cp{};
    cp.y = at<float>(h, pl.off_y);
    cp.final_norm = wt->final_norm; cp.w_cls = wt->w_cls; cp.b_cls = wt->b_cls;
    cp.logits = logits;
    cp.k = c.k; cp.d = d; cp.n_classes = c.n_classes; cp.pool_mean = c.pool == SP_POOL_MEAN;
    cp.eps = c.rms_eps;
    SP_TRY(launch_final_classifier(dt, cp, B, s));
  }
  if (!mark()) return SP_ERR_HIP;
#undef SP_TRY
  if (prof) ++h->n_profiled;
  return SP_OK;
}

SP_API size_t sp_probe_tap_bytes(const sp_probe_t* h, int tap, int32_t batch) {
  if (!h || batch < 0 || batch > h->cfg.max_batch) return 0;
  const sp_probe_config& c = h->cfg;
  const size_t M = (size_t)batch * c.k, e = h->plan.esz;
  switch (tap) {
    case SP_TAP_QKV: return (size_t)c.k * h->plan.nqkv * 4;
    case SP_TAP_ATTN: return M * c.n_q_heads * c.head_dim * e;
    case SP_TAP_A: return M * c.hidden * 4;
    case SP_TAP_Y: return M * c.hidden * 4;
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
  const int64_t total = h->n_profiled;
  const int64_t count = total < kMaxProfiled ? total : kMaxProfiled;
  for (int64_t f = total - count; f < total; ++f) {
    hipEvent_t* ev = &h->events[(size_t)(f % kMaxProfiled) * kEventsPerForward];
    if (hipEventSynchronize(ev[SP_N_STAGES]) != hipSuccess) return SP_ERR_HIP;
    for (int i = 0; i < n_stages; ++i) {
      float ms = 0.f;
      if (hipEventElapsedTime(&ms, ev[i], ev[i + 1]) != hipSuccess) return SP_ERR_HIP;
      stage_ms[i] += ms;
    }
  }
  if (n_forwards) *n_forwards = (int32_t)count;
  h->n_profiled = 0;
  return SP_OK;
}
