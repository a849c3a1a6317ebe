// Host runtime behind the C ABI of include/sp_probe.h: argument checks, split
// planning, workspace layout, the fp16 weight image and the launch sequence of
// one forward.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <deque>
#include <functional>
#include <mutex>
#include <new>
#include <vector>

#include "../../include/sp_probe.h"
#include "kernels.h"

#define SP_API extern "C" __attribute__((visibility("default")))

namespace {

using namespace sp;

// Profiling: a forward records one event at its start and one after every
// stage (the recursive forward: after every stage of every step), taken from a
// fixed pool used as a ring; the records of the last forwards that still fit
// are kept.
constexpr int kMaxProfiled = 256;
constexpr int kEventPool = kMaxProfiled * (SP_N_STAGES + 1);

// Compute units assumed where no device can be asked (host-only planning).
constexpr int kDefaultCus = 256;

// Workspace guards: every segment of the workspace is followed by kGuardBytes
// holding kGuardWord, written at init and checked by sp_probe_check_device_error.
constexpr size_t kGuardBytes = 256;
constexpr uint32_t kGuardWord = 0x5AFE6A4Du;
constexpr int kMaxGuards = 64;

// Words of the workspace's flag area: 0 debug validation (kernels skip work
// while it is non-zero), 1 status bits of any forward (kStatusSeqLen,
// kStatusRange), 2 guard check result, then the expected header of a weight
// image of this config.
constexpr int kFlagErr = 0, kFlagStatus = 1, kFlagGuard = 2, kFlagHeader = 8;

// fp16 weight image: a header, then the projection matrices as fp16, each
// segment 256-byte aligned: [Q; K; V] rows [(n_q + 2 n_kv) hd][d], W_o
// [d][n_q hd], W_gate [I][d], W_up [I][d], W_down [d][I].
constexpr uint32_t kImageMagic = 0x31504B53u;
constexpr int kHeaderWords = 8;
constexpr size_t kHeaderBytes = 256;

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }
int ilog2(int64_t x) { int r = 0; while ((int64_t(1) << r) < x) ++r; return r; }
bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

struct ImageLayout {
  size_t off_qkv, off_o, off_gate, off_up, off_down, total;
};

ImageLayout image_layout(const sp_probe_config& c) {
  const size_t d = c.hidden, hd = c.head_dim, I = c.intermediate;
  const size_t qkv = (size_t)(c.n_q_heads + 2 * c.n_kv_heads) * hd, qw = (size_t)c.n_q_heads * hd;
  ImageLayout L{};
  size_t o = kHeaderBytes;
  auto take = [&](size_t elems) { const size_t at = o; o = align256(o + elems * 2); return at; };
  L.off_qkv = take(qkv * d);
  L.off_o = take(d * qw);
  L.off_gate = take(I * d);
  L.off_up = take(I * d);
  L.off_down = take(d * I);
  L.total = o;
  return L;
}

void image_header(const sp_probe_config& c, uint32_t (&w)[kHeaderWords]) {
  const uint64_t total = image_layout(c).total;
  w[0] = kImageMagic;
  w[1] = (uint32_t)c.hidden;
  w[2] = (uint32_t)c.n_q_heads;
  w[3] = (uint32_t)c.n_kv_heads;
  w[4] = (uint32_t)c.head_dim;
  w[5] = (uint32_t)c.intermediate;
  w[6] = (uint32_t)(total & 0xffffffffu);
  w[7] = (uint32_t)(total >> 32);
}

// Attention launch shape for `rows` query rows per KV head.
struct AttnPlan {
  int rows, n_qgroups, r_alloc, split_len, max_splits;
  int tiles;  // 16-row query tiles per query group
  int waves;  // waves per workgroup (bf16 storage; tiles / waves query tiles per wave)
  int f16;    // bf16 storage: single fp16 products (matrix-core-bound shapes)
};

struct Plan {
  int group, max_tasks, ks, ks_rec, nqkv, esz, num_cus;
  int q_rows;    // query rows per (sequence, KV head) the one-pass query buffer holds
  AttnPlan rec;  // recursive steps: one soft row (G query rows) per KV head
  // workspace offsets (bytes)
  size_t off_u, off_qkv, off_q, off_ksoft, off_vsoft, off_q_lo, off_ksoft_lo, off_vsoft_lo,
      off_opart, off_ml, off_attn, off_a, off_w, off_s, off_y, off_err;
  // recursive steps only: per-sequence queries and soft keys/values, the fused
  // rows and their inputs
  size_t off_rq, off_rq_lo, off_rks, off_rks_lo, off_rvs, off_rvs_lo, off_rqkv, off_ru, off_rhn,
      off_ren, off_rce, off_rx, off_r3, off_rh0, off_rscale;
  size_t off_items, off_n_items;  // the attention's work list ([max_batch][splits] int32 pairs) and its length
  int items_splits;               // splits per sequence the work list has room for (the largest plan's)
  size_t off_gpart, gpart_bytes;  // split-K partial sums of the small-row projections
  size_t off_guard_tab;           // device table of the guard offsets
  size_t guard_off[kMaxGuards];
  int n_guards;
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
  if (c->n_q_heads > 4096 || c->max_batch > (1 << 20) || c->intermediate > (1 << 20))
    return SP_ERR_UNSUPPORTED;
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

AttnPlan attn_plan(const sp_probe_config& c, int rows, int num_cus) {
  AttnPlan a{};
  a.rows = rows;
  const int tiles = (rows + 15) / 16;
  if (c.dtype == SP_F32) {
    a.waves = 0;
    a.n_qgroups = 1;
    a.r_alloc = rows;
  } else {
    // 16-row query tiles per group: at most 12 (head_dim 128) or 16 (64), so
    // one workgroup reads each K/V tile for as many rows as fit (the 160 rows
    // of the 27B shape as one group of ten tiles: a second group would read
    // the cache twice); the sizes below are the planned ones (extra tiles are
    // padding).  Up to 6 tiles: one wave per tile.
    static const int kWaves[] = {1, 2, 3, 4, 5, 6, 8, 10, 12, 16};
    const int max_w = c.head_dim == 128 ? 12 : 16;
    const int groups = (tiles + max_w - 1) / max_w;
    const int per_group = (tiles + groups - 1) / groups;
    int w = max_w;
    for (int cand : kWaves)
      if (cand >= per_group) { w = cand; break; }
    a.tiles = w;
    a.waves = w;
    a.n_qgroups = (tiles + w - 1) / w;
    a.r_alloc = a.n_qgroups * w * 16;
    // Eight or more tiles per group (the 160 rows of the 27B shape, several
    // tasks): one wave per SIMD, each carrying 2-4 tiles, so every K/V fragment
    // read from LDS serves several tiles, with the K/V tiles converted to fp16
    // once in LDS and single fp16 products (27B shape: 2.7-2.8 ms against 5.0 ms
    // for ten waves of one tile and 4.8-5.5 ms for eight or five waves of two
    // tiles, which hold fewer waves per compute unit; hi + lo bf16 products at
    // 2-4 tiles per wave are matrix-core bound and gain nothing).
    if (w >= 8) {
      a.waves = 4;
      a.f16 = 1;
    }
  }
  if (c.split_len) {
    a.split_len = c.split_len;
  } else if (c.dtype == SP_BF16) {
    // Splits sized so that the attention grid at the full batch and length is
    // at least one round of resident workgroups, and at most a third of the longest
    // sequence: three splits for the longest sequences measured faster than
    // one, two or four on uniform and ragged batches alike, whether the grid
    // is one round or many.  At least 1024 tokens, a multiple of 256.
    const int64_t per_cu = attn_wgs_per_cu(c.head_dim, a.waves, (a.tiles + a.waves - 1) / a.waves);
    const int64_t slots = (int64_t)num_cus * std::max<int64_t>(per_cu, 1);
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
AttnPlan one_pass_plan(const sp_probe_config& c, int n_tasks, int num_cus) {
  const int group = c.n_q_heads / c.n_kv_heads;
  const int per_task = (c.flags & SP_FLAG_LAST_ROW_ONLY) ? 1 : c.k;
  return attn_plan(c, n_tasks * per_task * group, num_cus);
}

Plan make_plan(const sp_probe_config& c, int num_cus) {
  Plan p{};
  p.num_cus = num_cus;
  p.esz = c.dtype == SP_BF16 ? 2 : 4;
  p.group = c.n_q_heads / c.n_kv_heads;
  p.max_tasks = n_tasks_max(c);
  p.rec = attn_plan(c, p.group, num_cus);
  const int S = p.max_tasks * c.k;       // soft rows of the largest call
  p.ks = ((S + 31) / 32) * 32;
  p.ks_rec = ((c.k + 31) / 32) * 32;
  p.nqkv = (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  // split partials: the largest of every plan the handle can run
  size_t part_rows = (size_t)p.rec.max_splits * p.rec.r_alloc;
  p.q_rows = 0;
  p.items_splits = p.rec.max_splits;
  for (int t = 1; t <= p.max_tasks; ++t) {
    const AttnPlan a = one_pass_plan(c, t, num_cus);
    part_rows = std::max(part_rows, (size_t)a.max_splits * a.r_alloc);
    p.q_rows = std::max(p.q_rows, a.r_alloc);
    p.items_splits = std::max(p.items_splits, a.max_splits);
  }

  const size_t B = (size_t)c.max_batch, M = B * S, d = c.hidden, hd = c.head_dim;
  const size_t kv = (size_t)c.n_kv_heads, e = p.esz;
  size_t o = 0;
  // each segment is followed by a guard area
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align256(o + bytes);
    if (p.n_guards < kMaxGuards) p.guard_off[p.n_guards++] = o;
    o += kGuardBytes;
    return at;
  };
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
  p.off_opart = take(B * kv * part_rows * hd * e);  // fp16 O / l (bf16 storage) or fp32 O
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
  p.off_items = take(B * (size_t)p.items_splits * 8);
  p.off_n_items = take(4);
  // split-K partials: up to 512 rows of the widest product, and four slices of
  // a hidden-wide product on up to 1024 rows (o and down there split K)
  const size_t widest = std::max({(size_t)2 * c.intermediate, (size_t)p.nqkv, d});
  p.gpart_bytes = std::max(16 * 32 * widest, 4 * std::min<size_t>(M, 1024) * d) * 4;
  p.off_gpart = take(p.gpart_bytes);
  p.off_guard_tab = take(kMaxGuards * sizeof(uint64_t));
  p.total = o;
  return p;
}

// Compute units of the current device, or kDefaultCus when none can be asked.
int device_cus_or_default() {
  int count = 0, dev = 0;
  if (hipGetDeviceCount(&count) != hipSuccess || count < 1 || hipGetDevice(&dev) != hipSuccess)
    return kDefaultCus;
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
    return kDefaultCus;
  return cus;
}

}  // namespace

struct sp_probe {
  sp_probe_config cfg;
  Plan plan;
  int device, num_cus, n_xcd;
  char* ws;
  std::vector<hipEvent_t> events;  // kEventPool events (profiling mode), used as a ring
  struct Record { int start, marks; };
  std::deque<Record> records;      // forwards whose events are still in the pool, oldest first
  int cursor;                      // next free event of the pool
};

namespace {

// What a forward needs: the config, its plan, the workspace and the device's
// shape; the handle only for profiling events (nullable).
struct Ctx {
  const sp_probe_config* cfg;
  const Plan* plan;
  char* ws;
  int n_cus, n_xcd;
  sp_probe* prof;
};

Ctx ctx_of(sp_probe* h) { return Ctx{&h->cfg, &h->plan, h->ws, h->num_cus, h->n_xcd, h}; }

template <typename T>
T* at(const Ctx& x, size_t off) { return reinterpret_cast<T*>(x.ws + off); }

int check_device(int* num_cus, int* n_xcd) {
  int dev = 0, count = 0;
  if (hipGetDeviceCount(&count) != hipSuccess || count < 1) return SP_ERR_NO_DEVICE;
  if (hipGetDevice(&dev) != hipSuccess) return SP_ERR_NO_DEVICE;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return SP_ERR_NO_DEVICE;
  if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0) return SP_ERR_NO_DEVICE;
  if (num_cus) *num_cus = prop.multiProcessorCount > 0 ? prop.multiProcessorCount : kDefaultCus;
  if (n_xcd) {
    int x = 0;
    if (hipDeviceGetAttribute(&x, hipDeviceAttributeNumberOfXccs, dev) != hipSuccess || x < 1) x = 1;
    *n_xcd = x;
  }
  return SP_OK;
}

// Events for a forward of `marks` marks (contiguous in the pool; the oldest
// records they overlap are dropped).  nullptr when profiling is off.
hipEvent_t* prof_begin(sp_probe* h, int marks) {
  if (!h || h->events.empty() || marks > kEventPool) return nullptr;
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

int* status_word(const Ctx& x) { return at<int>(x, x.plan->off_err) + kFlagStatus; }

// A projection with the workspace's split-K scratch, the device shape and the status word.
hipError_t run_gemm(const Ctx& x, DType dt, Epilogue epi, GemmParams g, hipStream_t s) {
  g.part = at<float>(x, x.plan->off_gpart);
  g.part_bytes = x.plan->gpart_bytes;
  g.n_cus = x.n_cus;
  g.n_xcd = x.n_xcd;
  g.status = status_word(x);
  return launch_gemm(dt, epi, g, s);
}

// The head's projection matrices as the GEMMs read them: the caller's
// matrices, or the segments of an fp16 weight image (f16 = 1).
struct ProjW {
  const void *q, *k, *v, *o, *gate, *up, *down;
  int f16;
};

ProjW proj_weights(const sp_probe_config& c, const sp_probe_weights* wt) {
  ProjW w{};
  if (wt->packed) {
    const ImageLayout L = image_layout(c);
    const char* base = (const char*)wt->packed;
    const size_t d = c.hidden, hd = c.head_dim;
    w.q = base + L.off_qkv;
    w.k = (const char*)w.q + (size_t)c.n_q_heads * hd * d * 2;
    w.v = (const char*)w.k + (size_t)c.n_kv_heads * hd * d * 2;
    w.o = base + L.off_o;
    w.gate = base + L.off_gate;
    w.up = base + L.off_up;
    w.down = base + L.off_down;
    w.f16 = 1;
  } else {
    w = ProjW{wt->w_q, wt->w_k, wt->w_v, wt->w_o, wt->w_gate, wt->w_up, wt->w_down, 0};
  }
  return w;
}

// Host-side checks shared by the forwards; *noop is set for an empty batch.
int check_forward(const sp_probe_config& c, const Plan& pl, const sp_kv_cache* kv, const int32_t* seq_lens,
                  const int32_t* block_table, const void* soft_prompt, const sp_probe_weights* wt,
                  const float* logits, bool* noop) {
  *noop = false;
  if (!kv || !wt) return SP_ERR_INVALID_ARG;
  const int B = kv->batch;
  if (B < 0) return SP_ERR_INVALID_ARG;
  if (B > c.max_batch) return SP_ERR_CAPACITY;
  if (B == 0) { *noop = true; return SP_OK; }
  if (!seq_lens || !soft_prompt || !logits) return SP_ERR_INVALID_ARG;
  const void* always[5] = {wt->in_norm, wt->post_norm, wt->final_norm, wt->w_cls, soft_prompt};
  for (const void* q : always)
    if (!q || !aligned16(q)) return SP_ERR_INVALID_ARG;
  if (wt->packed) {
    // an fp16 image replaces the projection matrices (bf16 storage only)
    if (c.dtype != SP_BF16 || !aligned16(wt->packed)) return SP_ERR_INVALID_ARG;
  } else {
    const void* mats[7] = {wt->w_q, wt->w_k, wt->w_v, wt->w_o, wt->w_gate, wt->w_up, wt->w_down};
    for (const void* q : mats)
      if (!q || !aligned16(q)) return SP_ERR_INVALID_ARG;
  }
  if (wt->cls_rows && (wt->cls_vocab < 1 || ((uintptr_t)wt->cls_rows & 3))) return SP_ERR_INVALID_ARG;
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
  return SP_OK;
}

// Split-attention parameters over the caller's cache for one attention plan.
AttnParams attn_params(const Ctx& x, const AttnPlan& a, const sp_kv_cache* kv,
                       const int32_t* seq_lens, const int32_t* block_table, const int* errp,
                       const void* q, const void* q_lo, void* o_part, float2* ml_part) {
  const sp_probe_config& c = *x.cfg;
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
  ap.r_alloc = a.r_alloc; ap.n_qgroups = a.n_qgroups; ap.n_tiles = a.tiles;
  ap.bs_log2 = ilog2(kv->block_size); ap.mbps = kv->max_blocks_per_seq;
  ap.max_seq_len = c.max_seq_len; ap.split_len = a.split_len; ap.max_splits = a.max_splits;
  ap.num_cus = x.n_cus;
  ap.f16 = a.f16;
  ap.stages = 3;
  // bf16 path: the work list launch_work_list wrote for this plan
  ap.items = c.dtype == SP_BF16 ? at<int2>(x, x.plan->off_items) : nullptr;
  ap.n_items = c.dtype == SP_BF16 ? at<int>(x, x.plan->off_n_items) : nullptr;
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

GemmParams gemm_qkv(const sp_probe_config& c, const Plan& pl, const ProjW& pw, const void* a, void* out,
                    int M) {
  GemmParams g{};
  g.a = a;
  g.b[0] = pw.q; g.b[1] = pw.k; g.b[2] = pw.v;
  g.b_split0 = c.n_q_heads * c.head_dim;
  g.b_split1 = (c.n_q_heads + c.n_kv_heads) * c.head_dim;
  g.ldb = c.hidden;
  g.b_f16 = pw.f16;
  g.c = out;
  g.M = M; g.N = pl.nqkv; g.K = c.hidden; g.lda = c.hidden; g.ldc = pl.nqkv;
  return g;
}

GemmParams gemm_gate_up(const sp_probe_config& c, const ProjW& pw, const void* a, void* out, int M) {
  GemmParams g{};
  g.a = a;
  g.b[0] = pw.gate; g.b[1] = pw.up; g.b[2] = pw.up;
  g.b_split0 = g.b_split1 = 2 * c.intermediate;
  g.ldb = c.hidden;
  g.b_f16 = pw.f16;
  g.c = out;
  g.M = M; g.N = 2 * c.intermediate; g.K = c.hidden; g.lda = c.hidden; g.ldc = c.intermediate;
  return g;
}

// Debug mode with an fp16 weight image: its header must be this config's.
hipError_t check_image(const Ctx& x, const sp_probe_weights* wt, int* err, hipStream_t s) {
  if (!wt->packed) return hipSuccess;
  return launch_check_header((const uint32_t*)wt->packed, (const uint32_t*)err + kFlagHeader, kHeaderWords,
                             err, 64, s);
}

}  // namespace

SP_API size_t sp_probe_workspace_bytes(const sp_probe_config* cfg) {
  if (check_config(cfg) != SP_OK) return 0;
  return make_plan(*cfg, device_cus_or_default()).total;
}

SP_API const char* sp_probe_status_string(int status) {
  switch (status) {
    case SP_OK: return "SP_OK";
    case SP_ERR_INVALID_ARG: return "SP_ERR_INVALID_ARG: invalid argument";
    case SP_ERR_UNSUPPORTED: return "SP_ERR_UNSUPPORTED: configuration not supported";
    case SP_ERR_NO_DEVICE: return "SP_ERR_NO_DEVICE: no gfx950 HIP device";
    case SP_ERR_OUT_OF_MEMORY: return "SP_ERR_OUT_OF_MEMORY: workspace allocation failed";
    case SP_ERR_HIP: return "SP_ERR_HIP: HIP runtime or launch error";
    case SP_ERR_CAPACITY: return "SP_ERR_CAPACITY: batch exceeds max_batch, or the workspace exceeds the static scratch";
    case SP_ERR_DEVICE_DATA: return "SP_ERR_DEVICE_DATA: invalid seq_lens, block ids, class rows or weight image on the device";
    case SP_ERR_RANGE: return "SP_ERR_RANGE: an fp16 activation exceeded fp16's range";
    case SP_ERR_INTERNAL: return "SP_ERR_INTERNAL: a workspace guard word was overwritten, or the plan is inconsistent";
  }
  return "unknown status";
}

SP_API int sp_probe_init(const sp_probe_config* cfg, sp_probe_t** out) {
  if (!out) return SP_ERR_INVALID_ARG;
  *out = nullptr;
  int st = check_config(cfg);
  if (st != SP_OK) return st;
  int cus = 0, xcd = 0;
  st = check_device(&cus, &xcd);
  if (st != SP_OK) return st;
  sp_probe* h = new (std::nothrow) sp_probe();
  if (!h) return SP_ERR_OUT_OF_MEMORY;
  h->cfg = *cfg;
  h->num_cus = cus;
  h->n_xcd = xcd;
  h->plan = make_plan(*cfg, cus);
  h->cursor = 0;
  h->ws = nullptr;
  if (hipGetDevice(&h->device) != hipSuccess) { delete h; return SP_ERR_HIP; }
  if (hipMalloc(&h->ws, h->plan.total) != hipSuccess) { delete h; return SP_ERR_OUT_OF_MEMORY; }
  // Zero once: padded query rows and padded soft key/value slots stay zero for
  // the handle's lifetime (forwards only write the unpadded part).  Then the
  // guard words, their offset table and the expected weight-image header.
  const Plan& pl = h->plan;
  uint64_t offs[kMaxGuards];
  for (int i = 0; i < pl.n_guards; ++i) offs[i] = pl.guard_off[i];
  uint32_t hdr[kHeaderWords];
  image_header(*cfg, hdr);
  bool ok = hipMemset(h->ws, 0, pl.total) == hipSuccess;
  for (int i = 0; ok && i < pl.n_guards; ++i)
    ok = launch_fill_words((uint32_t*)(h->ws + pl.guard_off[i]), kGuardBytes / 4, kGuardWord, nullptr) == hipSuccess;
  ok = ok && hipMemcpy(h->ws + pl.off_guard_tab, offs, pl.n_guards * sizeof(uint64_t), hipMemcpyHostToDevice) == hipSuccess;
  ok = ok && hipMemcpy(h->ws + pl.off_err + kFlagHeader * 4, hdr, sizeof(hdr), hipMemcpyHostToDevice) == hipSuccess;
  ok = ok && hipDeviceSynchronize() == hipSuccess;
  if (!ok) {
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

namespace {
void write_plan(const AttnPlan& a, int32_t* split_len, int32_t* max_splits, int32_t* rows, int32_t* groups) {
  if (split_len) *split_len = a.split_len;
  if (max_splits) *max_splits = a.max_splits;
  if (rows) *rows = a.rows;
  if (groups) *groups = a.n_qgroups;
}
}  // namespace

SP_API int sp_probe_plan(const sp_probe_t* h, int32_t batch, int32_t* split_len, int32_t* max_splits,
                         int32_t* rows_per_kv_head, int32_t* query_groups) {
  if (!h || batch < 0) return SP_ERR_INVALID_ARG;
  write_plan(one_pass_plan(h->cfg, 1, h->num_cus), split_len, max_splits, rows_per_kv_head, query_groups);
  return SP_OK;
}

SP_API int sp_probe_plan_recursive(const sp_probe_t* h, int32_t batch, int32_t* split_len,
                                   int32_t* max_splits, int32_t* rows_per_kv_head,
                                   int32_t* query_groups) {
  if (!h || batch < 0) return SP_ERR_INVALID_ARG;
  write_plan(h->plan.rec, split_len, max_splits, rows_per_kv_head, query_groups);
  return SP_OK;
}

SP_API int sp_probe_plan_config(const sp_probe_config* cfg, int32_t num_cus, int32_t* split_len,
                                int32_t* max_splits, int32_t* rows_per_kv_head, int32_t* query_groups,
                                size_t* workspace_bytes) {
  const int st = check_config(cfg);
  if (st != SP_OK) return st;
  if (num_cus < 1 || num_cus > 65536) return SP_ERR_INVALID_ARG;
  write_plan(one_pass_plan(*cfg, 1, num_cus), split_len, max_splits, rows_per_kv_head, query_groups);
  if (workspace_bytes) *workspace_bytes = make_plan(*cfg, num_cus).total;
  return SP_OK;
}

SP_API size_t sp_probe_packed_bytes(const sp_probe_config* cfg) {
  if (check_config(cfg) != SP_OK || cfg->dtype != SP_BF16) return 0;
  return image_layout(*cfg).total;
}

SP_API int sp_probe_pack_weights(const sp_probe_config* cfg, const sp_probe_weights* weights, void* packed,
                                 size_t packed_bytes, void* stream) {
  int st = check_config(cfg);
  if (st != SP_OK) return st;
  if (cfg->dtype != SP_BF16) return SP_ERR_UNSUPPORTED;
  if (!weights || !packed || !aligned16(packed)) return SP_ERR_INVALID_ARG;
  const void* mats[7] = {weights->w_q, weights->w_k, weights->w_v, weights->w_o, weights->w_gate,
                         weights->w_up, weights->w_down};
  for (const void* q : mats)
    if (!q || !aligned16(q)) return SP_ERR_INVALID_ARG;
  const ImageLayout L = image_layout(*cfg);
  if (packed_bytes < L.total) return SP_ERR_INVALID_ARG;
  st = check_device(nullptr, nullptr);
  if (st != SP_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  const size_t d = cfg->hidden, hd = cfg->head_dim, I = cfg->intermediate;
  const size_t nq = (size_t)cfg->n_q_heads * hd, nkv = (size_t)cfg->n_kv_heads * hd;
  char* base = (char*)packed;
  uint32_t hdr[kHeaderWords];
  image_header(*cfg, hdr);
  const struct { const void* src; size_t off, n; } parts[7] = {
      {weights->w_q, L.off_qkv, nq * d},
      {weights->w_k, L.off_qkv + nq * d * 2, nkv * d},
      {weights->w_v, L.off_qkv + (nq + nkv) * d * 2, nkv * d},
      {weights->w_o, L.off_o, d * nq},
      {weights->w_gate, L.off_gate, I * d},
      {weights->w_up, L.off_up, I * d},
      {weights->w_down, L.off_down, d * I}};
  for (const auto& pt : parts)
    if (launch_bf16_to_f16(pt.src, base + pt.off, pt.n, s) != hipSuccess) return SP_ERR_HIP;
  for (int i = 0; i < kHeaderWords; ++i)
    if (launch_fill_words((uint32_t*)base + i, 1, hdr[i], s) != hipSuccess) return SP_ERR_HIP;
  return SP_OK;
}

#define SP_TRY(expr) do { if ((expr) != hipSuccess) return SP_ERR_HIP; } while (0)

namespace {

// The one-pass forward for n_tasks tasks (Sec. 3.2-3.3; one task is the plain
// probe): all tasks' soft rows share one pass over the cache.
int forward_one_pass(const Ctx& x, const sp_kv_cache* kv, const int32_t* seq_lens,
                     const int32_t* block_table, int n_tasks, const void* soft_prompt,
                     const sp_probe_weights* wt, float* logits, void* stream) {
  const sp_probe_config& c = *x.cfg;
  const Plan& pl = *x.plan;
  // ---- host-side checks: nothing is enqueued unless all pass
  bool noop = false;
  const int chk = check_forward(c, pl, kv, seq_lens, block_table, soft_prompt, wt, logits, &noop);
  if (chk != SP_OK) return chk;
  if (n_tasks < 1 || n_tasks > pl.max_tasks) return SP_ERR_INVALID_ARG;
  if (noop) return SP_OK;
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
  const AttnPlan ak = one_pass_plan(c, n_tasks, x.n_cus);
  const ProjW pw = proj_weights(c, wt);
  const bool debug = c.flags & SP_FLAG_DEBUG;
  int* err = at<int>(x, pl.off_err);
  int* status = status_word(x);
  const int* errp = debug ? err : nullptr;
  const int marks = SP_N_STAGES + 1;
  hipEvent_t* ev = prof_begin(x.prof, marks);
  int stage = 0;
  auto mark = [&]() -> bool { return !ev || hipEventRecord(ev[stage++], s) == hipSuccess; };

  if (debug) {
    ValidateParams vp{seq_lens, block_table, err, kv->num_blocks, kv->max_blocks_per_seq,
                      ilog2(kv->block_size), c.max_seq_len, wt->cls_rows, n_tasks * c.n_classes, wt->cls_vocab};
    SP_TRY(launch_validate(vp, B, s));
    SP_TRY(check_image(x, wt, err, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // stage 0: soft rows — RMSNorm, Q/K/V on the S distinct rows, RoPE per sequence
  SP_TRY(launch_rmsnorm_rows(dt, dt, at_dt, soft_prompt, d, wt->in_norm, nullptr,
                             at<void>(x, pl.off_u), d, S, d, c.rms_eps, status, s));
  SP_TRY(run_gemm(x, dt, kEpiStore, gemm_qkv(c, pl, pw, at<void>(x, pl.off_u), at<void>(x, pl.off_qkv), S), s));
  {
    RopeParams r{};
    r.qkv = at<float>(x, pl.off_qkv);
    r.seq_lens = seq_lens;
    r.err = errp;
    r.status = status;
    r.q = at<void>(x, pl.off_q);
    r.k_soft = at<void>(x, pl.off_ksoft);
    r.v_soft = at<void>(x, pl.off_vsoft);
    r.q_lo = at<void>(x, pl.off_q_lo);
    r.k_soft_lo = at<void>(x, pl.off_ksoft_lo);
    r.v_soft_lo = at<void>(x, pl.off_vsoft_lo);
    r.n_q = c.n_q_heads; r.n_kv = c.n_kv_heads; r.hd = hd; r.k = S; r.group = pl.group;
    r.r_alloc = ak.r_alloc; r.ks = pl.ks; r.max_seq_len = c.max_seq_len;
    r.step = 0; r.per_seq = 0;
    r.k_task = K; r.q_first = K - Kq; r.q_per_task = Kq;
    r.rope_base = c.rope_base;
    r.q_scale = (float)(1.4426950408889634 / __builtin_sqrt((double)hd));
    r.num_cus = x.n_cus;
    SP_TRY(launch_rope_scatter(dt, r, B, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // stage 1: split attention over the cached K/V, longest work items first
  const AttnParams ap = attn_params(x, ak, kv, seq_lens, block_table, errp, at<void>(x, pl.off_q),
                                    at<void>(x, pl.off_q_lo), at<void>(x, pl.off_opart),
                                    at<float2>(x, pl.off_ml));
  if (dt == kBF16) {
    if (ak.max_splits > pl.items_splits) return SP_ERR_INTERNAL;
    SP_TRY(launch_work_list(seq_lens, B, c.max_seq_len, ak.split_len, at<int2>(x, pl.off_items),
                            at<int>(x, pl.off_n_items), s));
    SP_TRY(launch_attention_bf16(ap, hd, ak.waves, B, s));
  } else {
    SP_TRY(launch_attention_f32(ap, hd, B, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // stage 2: merge the splits and each task's soft keys into the attention output rows
  {
    MergeParams mp{};
    mp.o_part = ap.o_part; mp.ml_part = ap.ml_part; mp.seq_lens = seq_lens; mp.err = errp;
    mp.q = ap.q; mp.q_lo = ap.q_lo;
    mp.k_soft = at<void>(x, pl.off_ksoft); mp.k_soft_lo = at<void>(x, pl.off_ksoft_lo);
    mp.v_soft = at<void>(x, pl.off_vsoft); mp.v_soft_lo = at<void>(x, pl.off_vsoft_lo);
    mp.out = at<void>(x, pl.off_attn);
    mp.status = status;
    mp.min_wgs = 4 * x.n_cus;
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
    GemmParams g = gemm_one(at<void>(x, pl.off_attn), qw, pw.o, qw, at<void>(x, pl.off_a), d, M, d, qw);
    g.b_f16 = pw.f16;
    g.r = (const char*)soft_prompt + (size_t)(K - Kq) * d * pl.esz;
    g.r_mod = R;
    g.r_ld = last_only ? K * d : d;
    SP_TRY(run_gemm(x, dt, kEpiResidRow, g, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // stage 4: w = RMSNorm(a; gamma_post)
  SP_TRY(launch_rmsnorm_rows(kF32, dt, at_dt, at<void>(x, pl.off_a), d, wt->post_norm, nullptr,
                             at<void>(x, pl.off_w), d, M, d, c.rms_eps, status, s));
  if (!mark()) return SP_ERR_HIP;

  // stage 5: s = silu(W_gate w) * (W_up w)
  SP_TRY(run_gemm(x, dt, kEpiSwiglu, gemm_gate_up(c, pw, at<void>(x, pl.off_w), at<void>(x, pl.off_s), M), s));
  if (!mark()) return SP_ERR_HIP;

  // stage 6: y = a + W_down s
  {
    GemmParams g = gemm_one(at<void>(x, pl.off_s), I, pw.down, I, at<void>(x, pl.off_y), d, M, d, I);
    g.b_f16 = pw.f16;
    g.r = at<void>(x, pl.off_a); g.r_ld = d;
    SP_TRY(run_gemm(x, dt, kEpiResidF32, g, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // stage 7: final RMSNorm, read-out, logits = W_cls pooled (+ b), per task
  {
    ClsParams cp{};
    cp.y = at<float>(x, pl.off_y);
    cp.final_norm = wt->final_norm; cp.w_cls = wt->w_cls; cp.b_cls = wt->b_cls;
    cp.cls_rows = wt->cls_rows; cp.err = errp;
    cp.logits = logits;
    cp.k = Kq; cp.n_tasks = n_tasks; cp.d = d; cp.n_classes = c.n_classes;
    cp.pool_mean = c.pool == SP_POOL_MEAN;
    cp.eps = c.rms_eps;
    SP_TRY(launch_final_classifier(dt, cp, B, s));
  }
  if (!mark()) return SP_ERR_HIP;
  if (ev) prof_commit(x.prof, marks);
  return SP_OK;
}

}  // namespace

SP_API int sp_probe_forward(sp_probe_t* h, const sp_kv_cache* kv, const int32_t* seq_lens,
                            const int32_t* block_table, const void* soft_prompt,
                            const sp_probe_weights* wt, float* logits, void* stream) {
  if (!h) return SP_ERR_INVALID_ARG;
  return forward_one_pass(ctx_of(h), kv, seq_lens, block_table, 1, soft_prompt, wt, logits, stream);
}

SP_API int sp_probe_forward_multi(sp_probe_t* h, const sp_kv_cache* kv, const int32_t* seq_lens,
                                  const int32_t* block_table, int32_t n_tasks, const void* soft_prompts,
                                  const sp_probe_weights* wt, float* logits, void* stream) {
  if (!h) return SP_ERR_INVALID_ARG;
  return forward_one_pass(ctx_of(h), kv, seq_lens, block_table, n_tasks, soft_prompts, wt, logits, stream);
}

SP_API int sp_probe_forward_recursive(sp_probe_t* h, const sp_kv_cache* kv, const int32_t* seq_lens,
                                      const int32_t* block_table, const void* soft_prompt,
                                      const void* hidden_last, const sp_probe_fusion* fusion,
                                      const sp_probe_weights* wt, float* logits, void* stream) {
  if (!h) return SP_ERR_INVALID_ARG;
  const Ctx x = ctx_of(h);
  const sp_probe_config& c = *x.cfg;
  const Plan& pl = *x.plan;
  // ---- host-side checks: nothing is enqueued unless all pass
  bool noop = false;
  const int chk = check_forward(c, pl, kv, seq_lens, block_table, soft_prompt, wt, logits, &noop);
  if (chk != SP_OK || noop) return chk;
  if (!fusion || !hidden_last || !aligned16(hidden_last)) return SP_ERR_INVALID_ARG;
  const void* fptr[3] = {fusion->fc_norm_hidden, fusion->fc_norm_embed, fusion->w_fc};
  for (const void* q : fptr)
    if (!q || !aligned16(q)) return SP_ERR_INVALID_ARG;
  const bool eagle3 = fusion->w_hidden_fuse != nullptr;
  if (eagle3 && !aligned16(fusion->w_hidden_fuse)) return SP_ERR_INVALID_ARG;
  const AttnPlan& rp = pl.rec;
  const int B = kv->batch, K = c.k;
  const ProjW pw = proj_weights(c, wt);

  hipStream_t s = (hipStream_t)stream;
  const DType dt = c.dtype == SP_BF16 ? kBF16 : kF32;
  const DType at_dt = c.dtype == SP_BF16 ? kF16 : kF32;
  const int d = c.hidden, hd = c.head_dim, I = c.intermediate, qw = c.n_q_heads * hd;
  const size_t esz = pl.esz;  // bytes of a storage element and of an activation element
  const int64_t ld_steps = (int64_t)K * d;  // row stride of the [B][k][d] step buffers
  const bool debug = c.flags & SP_FLAG_DEBUG;
  int* err = at<int>(x, pl.off_err);
  int* status = status_word(x);
  const int* errp = debug ? err : nullptr;
  const int marks = SP_N_STAGES * K + 1;
  hipEvent_t* ev = prof_begin(x.prof, marks);
  int mk = 0;
  auto mark = [&]() -> bool { return !ev || hipEventRecord(ev[mk++], s) == hipSuccess; };

  char* x_all = at<char>(x, pl.off_rx);   // fused rows x_t: fp32 [B][k][d]
  char* a_all = at<char>(x, pl.off_a);    // a_t: fp32 [B][k][d]
  char* y_all = at<char>(x, pl.off_y);    // y_t: fp32 [B][k][d]
  char* o_all = at<char>(x, pl.off_attn); // attention output: [B][k][n_q hd]
  void* hn = at<void>(x, pl.off_rhn);     // RMSNorm of the hidden state entering a step
  const void* w_fc_embed = (const char*)fusion->w_fc + (size_t)d * esz;  // columns d..2d-1

  if (debug) {
    ValidateParams vp{seq_lens, block_table, err, kv->num_blocks, kv->max_blocks_per_seq,
                      ilog2(kv->block_size), c.max_seq_len, wt->cls_rows, c.n_classes, wt->cls_vocab};
    SP_TRY(launch_validate(vp, B, s));
    SP_TRY(check_image(x, wt, err, s));
  }
  if (!mark()) return SP_ERR_HIP;

  // The soft-prompt half of the fusion does not depend on the sequence:
  // c_t = W_fc[:, d:] RMSNorm(e_t; gamma_e) for the k steps, once.
  SP_TRY(launch_rmsnorm_rows(dt, dt, at_dt, soft_prompt, d, fusion->fc_norm_embed, nullptr,
                             at<void>(x, pl.off_ren), d, K, d, c.rms_eps, status, s));
  SP_TRY(run_gemm(x, dt, kEpiStore, gemm_one(at<void>(x, pl.off_ren), d, w_fc_embed, 2 * d,
                                             at<void>(x, pl.off_rce), d, K, d, d), s));
  if (!eagle3) {
    // the first step's hidden state is the base model's last one
    SP_TRY(launch_rmsnorm_rows(dt, dt, at_dt, hidden_last, d, fusion->fc_norm_hidden, nullptr, hn, d,
                               B, d, c.rms_eps, status, s));
  } else {
    // Eagle3: the first step's hidden state is W [h_low; h_mid; h_high]; on the
    // bf16 path the three states enter the MFMA as fp16 rows scaled by a power
    // of two (their range can exceed fp16's) and the product is scaled back
    float* h0 = at<float>(x, pl.off_rh0);
    if (dt == kBF16) {
      SP_TRY(launch_scale_rows_f16(hidden_last, 3 * d, at<void>(x, pl.off_r3), at<float>(x, pl.off_rscale),
                                   B, 3 * d, s));
      GemmParams g = gemm_one(at<void>(x, pl.off_r3), 3 * d, fusion->w_hidden_fuse, 3 * d, h0, d, B, d, 3 * d);
      g.r = at<float>(x, pl.off_rscale);
      SP_TRY(run_gemm(x, dt, kEpiRowScale, g, s));
    } else {
      SP_TRY(run_gemm(x, dt, kEpiStore, gemm_one(hidden_last, 3 * d, fusion->w_hidden_fuse, 3 * d, h0, d,
                                                 B, d, 3 * d), s));
    }
    SP_TRY(launch_rmsnorm_rows(kF32, dt, at_dt, h0, d, fusion->fc_norm_hidden, nullptr, hn, d, B, d,
                               c.rms_eps, status, s));
  }

  // the attention of every step runs the same work list, longest items first
  if (dt == kBF16) {
    if (pl.rec.max_splits > pl.items_splits) return SP_ERR_INTERNAL;
    SP_TRY(launch_work_list(seq_lens, B, c.max_seq_len, pl.rec.split_len, at<int2>(x, pl.off_items),
                            at<int>(x, pl.off_n_items), s));
  }

  for (int t = 0; t < K; ++t) {
    // stage 0: x_t = W_fc[:, :d] RMSNorm(h; gamma_h) + c_t, its RMSNorm, Q/K/V, RoPE at N_b + t
    {
      GemmParams g = gemm_one(hn, d, fusion->w_fc, 2 * d, x_all + (size_t)t * d * 4, (int)ld_steps,
                              B, d, d);
      g.r = at<char>(x, pl.off_rce) + (size_t)t * d * 4; g.r_ld = 0;
      SP_TRY(run_gemm(x, dt, kEpiResidF32, g, s));
    }
    SP_TRY(launch_rmsnorm_rows(kF32, dt, at_dt, x_all + (size_t)t * d * 4, ld_steps, wt->in_norm,
                               nullptr, at<void>(x, pl.off_ru), d, B, d, c.rms_eps, status, s));
    SP_TRY(run_gemm(x, dt, kEpiStore, gemm_qkv(c, pl, pw, at<void>(x, pl.off_ru), at<void>(x, pl.off_rqkv), B), s));
    {
      RopeParams r{};
      r.qkv = at<float>(x, pl.off_rqkv);
      r.seq_lens = seq_lens;
      r.err = errp;
      r.status = status;
      r.q = at<void>(x, pl.off_rq);
      r.k_soft = at<void>(x, pl.off_rks);
      r.v_soft = at<void>(x, pl.off_rvs);
      r.q_lo = at<void>(x, pl.off_rq_lo);
      r.k_soft_lo = at<void>(x, pl.off_rks_lo);
      r.v_soft_lo = at<void>(x, pl.off_rvs_lo);
      r.n_q = c.n_q_heads; r.n_kv = c.n_kv_heads; r.hd = hd; r.k = 1; r.group = pl.group;
      r.r_alloc = rp.r_alloc; r.ks = pl.ks_rec; r.max_seq_len = c.max_seq_len;
      r.step = t; r.per_seq = 1;
      r.k_task = 1; r.q_first = 0; r.q_per_task = 1;
      r.rope_base = c.rope_base;
      r.q_scale = (float)(1.4426950408889634 / __builtin_sqrt((double)hd));
      r.num_cus = x.n_cus;
      SP_TRY(launch_rope_scatter(dt, r, B, s));
    }
    if (!mark()) return SP_ERR_HIP;

    // stage 1: split attention of the step's G query rows per KV head over the cache
    const AttnParams ap = attn_params(x, rp, kv, seq_lens, block_table, errp, at<void>(x, pl.off_rq),
                                      at<void>(x, pl.off_rq_lo), at<void>(x, pl.off_opart),
                                      at<float2>(x, pl.off_ml));
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
      mp.k_soft = at<void>(x, pl.off_rks); mp.k_soft_lo = at<void>(x, pl.off_rks_lo);
      mp.v_soft = at<void>(x, pl.off_rvs); mp.v_soft_lo = at<void>(x, pl.off_rvs_lo);
      mp.out = o_all;
      mp.status = status;
      mp.min_wgs = 4 * x.n_cus;
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
      GemmParams g = gemm_one(o_all + (size_t)t * qw * esz, K * qw, pw.o, qw,
                              a_all + (size_t)t * d * 4, (int)ld_steps, B, d, qw);
      g.b_f16 = pw.f16;
      g.r = x_all + (size_t)t * d * 4; g.r_ld = (int)ld_steps;
      SP_TRY(run_gemm(x, dt, kEpiResidF32, g, s));
    }
    if (!mark()) return SP_ERR_HIP;

    // stage 4: w = RMSNorm(a_t; gamma_post)
    SP_TRY(launch_rmsnorm_rows(kF32, dt, at_dt, a_all + (size_t)t * d * 4, ld_steps, wt->post_norm,
                               nullptr, at<void>(x, pl.off_w), d, B, d, c.rms_eps, status, s));
    if (!mark()) return SP_ERR_HIP;

    // stage 5: s = silu(W_gate w) * (W_up w)
    SP_TRY(run_gemm(x, dt, kEpiSwiglu, gemm_gate_up(c, pw, at<void>(x, pl.off_w), at<void>(x, pl.off_s), B), s));
    if (!mark()) return SP_ERR_HIP;

    // stage 6: y_t = a_t + W_down s
    {
      GemmParams g = gemm_one(at<void>(x, pl.off_s), I, pw.down, I, y_all + (size_t)t * d * 4,
                              (int)ld_steps, B, d, I);
      g.b_f16 = pw.f16;
      g.r = a_all + (size_t)t * d * 4; g.r_ld = (int)ld_steps;
      SP_TRY(run_gemm(x, dt, kEpiResidF32, g, s));
    }
    if (!mark()) return SP_ERR_HIP;

    // stage 7: the step's output f_t = RMSNorm(y_t; gamma_final) is the next
    // step's hidden state, which enters it as RMSNorm(f_t; gamma_h); after the
    // last step, the read-out and the classifier
    if (t + 1 < K) {
      SP_TRY(launch_rmsnorm_rows(kF32, dt, at_dt, y_all + (size_t)t * d * 4, ld_steps, wt->final_norm,
                                 fusion->fc_norm_hidden, hn, d, B, d, c.rms_eps, status, s));
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
  if (ev) prof_commit(x.prof, marks);
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
  const Plan& pl = h->plan;
  int* flags = reinterpret_cast<int*>(h->ws + pl.off_err);
  if (launch_check_guards(h->ws, reinterpret_cast<const uint64_t*>(h->ws + pl.off_guard_tab), pl.n_guards,
                          (int)(kGuardBytes / 4), kGuardWord, flags + kFlagGuard, 1, s) != hipSuccess)
    return SP_ERR_HIP;
  if (hipStreamSynchronize(s) != hipSuccess) return SP_ERR_HIP;
  int val[3] = {0, 0, 0};
  if (hipMemcpy(val, flags, sizeof(val), hipMemcpyDeviceToHost) != hipSuccess) return SP_ERR_HIP;
  if (val[0] || val[1] || val[2]) {
    if (hipMemset(flags, 0, sizeof(val)) != hipSuccess || hipDeviceSynchronize() != hipSuccess)
      return SP_ERR_HIP;
  }
  if (val[2]) return SP_ERR_INTERNAL;
  if (val[0] || (val[1] & kStatusSeqLen)) return SP_ERR_DEVICE_DATA;
  if (val[1] & kStatusRange) return SP_ERR_RANGE;
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

// ---------------------------------------------------------------- forward without allocation
// For callers that cannot allocate (code under graph capture, serving loops,
// harnesses that forbid hipMalloc): the workspace is a file-scope device array
// of kScratchBytes, one per device the library runs on, held until the process
// ends.  Host code must use its device address from hipGetSymbolAddress, taken
// once per device with that device current; the array's name is not a device
// address on the host.
namespace {

constexpr size_t kScratchBytes = size_t(64) << 20;
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

struct ScratchDev {
  std::once_flag once;
  int status;   // SP_OK once set up
  char* ptr;    // device address of this device's scratch array
  int num_cus, n_xcd;
};
ScratchDev g_scratch[kMaxDevices];

void setup_scratch(ScratchDev& sd) {
  int cus = 0, xcd = 0;
  sd.status = check_device(&cus, &xcd);
  if (sd.status != SP_OK) return;
  void* p = nullptr;
  if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
    sd.status = SP_ERR_HIP;
    return;
  }
  sd.ptr = static_cast<char*>(p);
  sd.num_cus = cus;
  sd.n_xcd = xcd;
}

}  // namespace

SP_API int sp_probe_forward_noalloc(const sp_probe_config* cfg, const sp_kv_cache* kv, const int32_t* seq_lens,
                                    const int32_t* block_table, const void* soft_prompt,
                                    const sp_probe_weights* weights, float* logits, void* stream) {
  int st = check_config(cfg);
  if (st != SP_OK) return st;
  if (cfg->flags & (SP_FLAG_DEBUG | SP_FLAG_PROFILE)) return SP_ERR_UNSUPPORTED;
  int dev = 0, count = 0;
  if (hipGetDeviceCount(&count) != hipSuccess || count < 1 || hipGetDevice(&dev) != hipSuccess)
    return SP_ERR_NO_DEVICE;
  if (dev < 0 || dev >= kMaxDevices) return SP_ERR_UNSUPPORTED;
  ScratchDev& sd = g_scratch[dev];
  std::call_once(sd.once, setup_scratch, std::ref(sd));
  if (sd.status != SP_OK) return sd.status;
  const Plan pl = make_plan(*cfg, sd.num_cus);
  if (pl.total > kScratchBytes) return SP_ERR_CAPACITY;
  const Ctx x{cfg, &pl, sd.ptr, sd.num_cus, sd.n_xcd, nullptr};
  // host checks first: on error nothing is enqueued
  bool noop = false;
  st = check_forward(*cfg, pl, kv, seq_lens, block_table, soft_prompt, weights, logits, &noop);
  if (st != SP_OK || noop) return st;
  // The array keeps the last call's contents (possibly of another config):
  // clear what a forward expects to start at zero, the padded query rows and
  // soft key/value slots and the flag words, with a fill kernel.
  hipStream_t s = (hipStream_t)stream;
  const size_t zero_from[] = {pl.off_q, pl.off_ksoft, pl.off_vsoft, pl.off_q_lo, pl.off_ksoft_lo,
                              pl.off_vsoft_lo, pl.off_err};
  const size_t zero_to[] = {pl.off_ksoft, pl.off_vsoft, pl.off_q_lo, pl.off_ksoft_lo, pl.off_vsoft_lo,
                            pl.off_opart, pl.off_err + 256};
  for (int i = 0; i < 7; ++i)
    if (zero_to[i] > zero_from[i] &&
        launch_fill_words((uint32_t*)(sd.ptr + zero_from[i]), (zero_to[i] - zero_from[i]) / 4, 0u, s) != hipSuccess)
      return SP_ERR_HIP;
  return forward_one_pass(x, kv, seq_lens, block_table, 1, soft_prompt, weights, logits, stream);
}
