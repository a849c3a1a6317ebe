// Host-side check of the runtime (config checks, planning, workspace layout,
// argument checks and the launch sequence of every forward), built with
// AddressSanitizer and UndefinedBehaviorSanitizer and run on the CPU.
//
// The runtime source is compiled into this program; the kernel launchers it
// calls are replaced by recorders that never touch memory.  Each recorder
// computes the workspace bytes its kernel would read or write from its
// parameters and checks that they lie inside the workspace and overlap none of
// its guard areas, and checks the index invariants the kernels rely on (soft
// slots inside the key buffer, query rows inside the padded tiles, output rows
// inside their buffer).  The forwards run over the probe's workloads, their
// task counts and row pruning, the recursive form, the fp16 weight image, and
// seeded random shapes, at several compute-unit counts.
#include "../../paper_2608_28099_amd/csrc/runtime.hip"

#include <cstdio>
#include <cstdlib>
#include <random>
#include <string>

namespace {

struct Checker {
  const char* ws = nullptr;
  const Plan* plan = nullptr;
  std::string where;
  long failures = 0, checks = 0;

  void fail(const std::string& msg) {
    if (failures < 40) std::fprintf(stderr, "FAIL [%s] %s\n", where.c_str(), msg.c_str());
    ++failures;
  }
  void expect(bool ok, const std::string& msg) {
    ++checks;
    if (!ok) fail(msg);
  }
  // Bytes [p, p + n) must, if p is inside the workspace, end inside it and miss every guard.
  void range(const void* p, size_t n, const char* what) {
    ++checks;
    if (!ws || !p || n == 0) return;
    const char* c = static_cast<const char*>(p);
    if (c < ws || c >= ws + plan->total) return;  // caller memory
    const size_t lo = (size_t)(c - ws), hi = lo + n;
    if (hi > plan->total) {
      fail(std::string(what) + ": past the workspace end");
      return;
    }
    for (int i = 0; i < plan->n_guards; ++i) {
      const size_t g0 = plan->guard_off[i], g1 = g0 + kGuardBytes;
      if (lo < g1 && g0 < hi) {
        fail(std::string(what) + ": overlaps guard " + std::to_string(i));
        return;
      }
    }
  }
};
Checker g;

size_t dsize(DType t) { return t == kF32 ? 4 : 2; }

}  // namespace

namespace sp {

hipError_t launch_rmsnorm_rows(DType in_dt, DType gain_dt, DType out_dt, const void* x, int64_t ld_x,
                               const void* gain, const void* gain2, void* out, int64_t ld_out, int rows, int d,
                               float eps, int* status, hipStream_t) {
  (void)gain_dt; (void)gain; (void)gain2; (void)eps;
  g.expect(rows >= 0 && d > 0 && d % 4 == 0 && d <= 16384, "rmsnorm shape");
  if (rows <= 0) return hipSuccess;
  g.range(x, ((size_t)(rows - 1) * ld_x + d) * dsize(in_dt), "rmsnorm in");
  g.range(out, ((size_t)(rows - 1) * ld_out + d) * dsize(out_dt), "rmsnorm out");
  g.range(status, 4, "status");
  return hipSuccess;
}

hipError_t launch_rope_scatter(DType dt, const RopeParams& p, int batch, hipStream_t) {
  const size_t e = dsize(dt), hd = p.hd;
  g.expect(p.k >= 1 && p.k_task >= 1 && p.q_per_task >= 1 && p.q_first >= 0 && p.q_first + p.q_per_task == p.k_task,
           "rope task layout");
  // every soft slot written lies inside the key buffer, every query row inside its tile
  g.expect(p.step + p.k <= p.ks, "rope: soft slot past ks");
  for (int j = 0; j < p.k; ++j) {
    const int jj = j % p.k_task;
    if (jj < p.q_first) continue;
    const int qi = (j / p.k_task) * p.q_per_task + jj - p.q_first;
    g.expect((qi + 1) * p.group <= p.r_alloc, "rope: query row past r_alloc");
  }
  const size_t qkv_rows = (size_t)(p.per_seq ? (size_t)(batch - 1) * p.k : 0) + p.k;
  g.range(p.qkv, qkv_rows * (p.n_q + 2 * p.n_kv) * hd * 4, "rope qkv");
  const size_t q = (size_t)batch * p.n_kv * p.r_alloc * hd * e;
  const size_t ks = (size_t)batch * p.n_kv * p.ks * hd * e;
  const size_t vs = (size_t)(p.per_seq ? batch : 1) * p.n_kv * p.ks * hd * e;
  g.range(p.q, q, "rope q");
  g.range(p.k_soft, ks, "rope k_soft");
  g.range(p.v_soft, vs, "rope v_soft");
  if (dt == kBF16) {
    g.range(p.q_lo, q, "rope q_lo");
    g.range(p.k_soft_lo, ks, "rope k_soft_lo");
    g.range(p.v_soft_lo, vs, "rope v_soft_lo");
  }
  g.range(p.status, 4, "status");
  return hipSuccess;
}

hipError_t launch_scale_rows_f16(const void* x, int64_t ld_x, void* out, float* inv_scale, int rows, int cols,
                                 hipStream_t) {
  g.range(x, ((size_t)(rows - 1) * ld_x + cols) * 2, "scale rows in");
  g.range(out, (size_t)rows * cols * 2, "scale rows out");
  g.range(inv_scale, (size_t)rows * 4, "scale rows factors");
  return hipSuccess;
}

static void attn_common(const AttnParams& p, int hd, int batch, size_t e) {
  g.expect(p.rows <= p.r_alloc, "attention rows past r_alloc");
  g.expect(p.split_len > 0 && (int64_t)p.max_splits * p.split_len >= p.max_seq_len, "splits cover max_seq_len");
  g.expect(p.num_cus >= 1, "attention: compute units");
  const size_t rows = (size_t)batch * p.n_kv * p.r_alloc;
  g.range(p.q, rows * hd * e, "attention q");
  if (e == 2) g.range(p.q_lo, rows * hd * e, "attention q_lo");
  g.range(p.o_part, rows * p.max_splits * hd * e, "attention o_part");  // fp16 (bf16 path) or fp32
  g.range(p.ml_part, rows * p.max_splits * 8, "attention ml_part");
  if (p.items) {
    g.range(p.items, (size_t)batch * p.max_splits * 8, "attention work list");
    g.range(p.n_items, 4, "attention work-list length");
  }
}

hipError_t launch_attention_bf16(const AttnParams& p, int hd, int waves, int batch, hipStream_t) {
  g.expect(p.n_qgroups * p.n_tiles * 16 == p.r_alloc && p.n_tiles >= waves && p.n_tiles <= 4 * waves,
           "attention tiles");
  g.expect(p.split_len % 32 == 0, "split_len multiple of the unit");
  attn_common(p, hd, batch, 2);
  return hipSuccess;
}

hipError_t launch_work_list(const int* seq_lens, int batch, int max_seq_len, int split_len, int2* items, int* count,
                            hipStream_t) {
  (void)seq_lens;
  g.expect(split_len > 0, "work list: split_len");
  g.range(items, (size_t)batch * ((max_seq_len + split_len - 1) / split_len > 0 ? (max_seq_len + split_len - 1) / split_len : 1) * 8,
          "work list");
  g.range(count, 4, "work-list length");
  return hipSuccess;
}

hipError_t launch_attention_f32(const AttnParams& p, int hd, int batch, hipStream_t) {
  g.expect(p.rows <= 64, "fp32 attention rows");
  attn_common(p, hd, batch, 4);
  return hipSuccess;
}

hipError_t launch_merge(DType dt, const MergeParams& p, int batch, hipStream_t) {
  const size_t e = dsize(dt), hd = p.hd;
  g.expect(p.rows % p.group == 0 && (p.rows / p.group) % p.q_per_task == 0, "merge row layout");
  g.expect(p.q_first + p.q_per_task + p.step <= p.ks && p.q_first + p.q_per_task + p.step <= 64,
           "merge: key window past ks");
  g.expect(p.out_off + p.rows / p.group <= p.out_rows, "merge: output row past out_rows");
  g.expect(p.min_wgs >= 1, "merge: minimum workgroups");
  const size_t rows = (size_t)batch * p.n_kv * p.r_alloc;
  g.range(p.o_part, rows * p.max_splits * hd * e, "merge o_part");
  g.range(p.ml_part, rows * p.max_splits * 8, "merge ml_part");
  g.range(p.q, rows * hd * e, "merge q");
  g.range(p.k_soft, (size_t)batch * p.n_kv * p.ks * hd * e, "merge k_soft");
  g.range(p.v_soft, (size_t)(p.per_seq ? batch : 1) * p.n_kv * p.ks * hd * e, "merge v_soft");
  g.range(p.out, (size_t)batch * p.out_rows * p.n_q * hd * e, "merge out");
  g.range(p.status, 4, "status");
  return hipSuccess;
}

hipError_t launch_gemm(DType dt, Epilogue epi, const GemmParams& p, hipStream_t) {
  if (p.M <= 0) return hipSuccess;
  g.expect(!p.b_f16 || dt == kBF16, "fp16 image on an fp32 config");
  g.expect(p.N > 0 && p.K > 0 && p.lda >= p.K && p.ldb >= p.K, "gemm shape");
  const size_t ea = dt == kF32 ? 4 : 2;
  const int n_out = epi == kEpiSwiglu ? p.N / 2 : p.N;
  g.expect(p.ldc >= n_out, "gemm ldc");
  g.range(p.a, ((size_t)(p.M - 1) * p.lda + p.K) * ea, "gemm a");
  const size_t ec = (epi == kEpiSwiglu && dt == kBF16) ? 2 : 4;
  g.range(p.c, ((size_t)(p.M - 1) * p.ldc + n_out) * ec, "gemm c");
  if (epi == kEpiResidF32)
    g.range(p.r, (p.r_ld ? (size_t)(p.M - 1) * p.r_ld + p.N : (size_t)p.N) * 4, "gemm residual");
  if (epi == kEpiResidRow) {
    g.expect(p.r_mod >= 1, "gemm residual rows");
    g.range(p.r, ((size_t)(std::min(p.M, p.r_mod) - 1) * p.r_ld + p.N) * ea, "gemm residual row");
  }
  if (epi == kEpiRowScale) g.range(p.r, (size_t)p.M * 4, "gemm row scales");
  g.range(p.part, p.part_bytes, "gemm split-K scratch");
  g.range(p.status, 4, "status");
  g.expect(p.n_cus >= 1 && p.n_xcd >= 1, "gemm device shape");
  return hipSuccess;
}

hipError_t launch_final_classifier(DType dt, const ClsParams& p, int batch, hipStream_t) {
  (void)dt;
  g.range(p.y, (size_t)batch * p.n_tasks * p.k * p.d * 4, "classifier y");
  return hipSuccess;
}

hipError_t launch_validate(const ValidateParams& p, int batch, hipStream_t) {
  (void)batch;
  g.range(p.err, 4, "validate flag");
  return hipSuccess;
}

hipError_t launch_fill_words(uint32_t* p, size_t n, uint32_t value, hipStream_t) {
  (void)value;
  g.range(p, n * 4, "fill");
  return hipSuccess;
}

hipError_t launch_check_guards(const char* base, const uint64_t* offs, int n_guards, int words, uint32_t value,
                               int* flag, int bit, hipStream_t) {
  (void)base; (void)offs; (void)n_guards; (void)words; (void)value; (void)flag; (void)bit;
  return hipSuccess;
}

hipError_t launch_bf16_to_f16(const void* src, void* dst, size_t n, hipStream_t) {
  (void)src; (void)dst; (void)n;
  return hipSuccess;
}

hipError_t launch_check_header(const uint32_t* image, const uint32_t* expect, int n_words, int* flag, int bit,
                               hipStream_t) {
  (void)image; (void)bit;
  g.range(expect, (size_t)n_words * 4, "expected header");
  g.range(flag, 4, "header flag");
  return hipSuccess;
}

}  // namespace sp

namespace {

// Fake device addresses for caller buffers: distinct, 256-byte aligned, never dereferenced.
const void* fake(uintptr_t i) { return reinterpret_cast<const void*>((uintptr_t)0x7f0000000000ull + i * 0x10000000ull); }

sp_probe_config make_cfg(int d, int nq, int nkv, int hd, int I, int k, int C, int dtype, int pool, int B, int N,
                         int flags, int tasks, int split_len) {
  sp_probe_config c{};
  c.hidden = d; c.n_q_heads = nq; c.n_kv_heads = nkv; c.head_dim = hd; c.intermediate = I; c.k = k;
  c.n_classes = C; c.dtype = dtype; c.pool = pool; c.rms_eps = 1e-6f; c.rope_base = 10000.0;
  c.max_batch = B; c.max_seq_len = N; c.split_len = split_len; c.flags = flags; c.max_tasks = tasks;
  return c;
}

void run_forwards(const sp_probe_config& cfg, int cus, const std::string& name) {
  if (check_config(&cfg) != SP_OK) return;
  sp_probe h{};
  h.cfg = cfg;
  h.num_cus = cus;
  h.n_xcd = 8;
  h.plan = make_plan(cfg, cus);
  h.cursor = 0;
  // the workspace is never dereferenced: a fake device range
  h.ws = reinterpret_cast<char*>((uintptr_t)0x100000000000ull);
  g.ws = h.ws;
  g.plan = &h.plan;
  // layout: segments in order, each followed by its guard, all inside total
  for (int i = 0; i < h.plan.n_guards; ++i)
    g.expect(h.plan.guard_off[i] + kGuardBytes <= h.plan.total && h.plan.guard_off[i] % 256 == 0, "guard placement");
  sp_kv_cache kv{};
  kv.k_base = fake(1); kv.v_base = fake(2);
  kv.block_size = 16;
  kv.max_blocks_per_seq = std::max(1, (cfg.max_seq_len + 15) / 16);
  kv.num_blocks = (int64_t)cfg.max_batch * kv.max_blocks_per_seq + 8;
  const int64_t tile = 16 * cfg.head_dim;
  kv.k_stride_head = kv.v_stride_head = tile;
  kv.k_stride_block = kv.v_stride_block = tile * cfg.n_kv_heads;
  sp_probe_weights wt{};
  const void** slots[] = {&wt.in_norm, &wt.w_q, &wt.w_k, &wt.w_v, &wt.w_o, &wt.post_norm, &wt.w_gate,
                          &wt.w_up, &wt.w_down, &wt.final_norm, &wt.w_cls};
  for (int i = 0; i < 11; ++i) *slots[i] = fake(10 + i);
  sp_probe_fusion fu{fake(30), fake(31), fake(32), nullptr};
  const int32_t* lens = (const int32_t*)fake(40);
  const int32_t* table = (const int32_t*)fake(41);
  float* logits = (float*)fake(42);
  const void* soft = fake(43);
  const void* hidden = fake(44);
  const int batches[] = {cfg.max_batch, std::max(1, cfg.max_batch / 2), 1};
  for (int packed = 0; packed < 2; ++packed) {
    if (packed && cfg.dtype != SP_BF16) continue;
    wt.packed = packed ? fake(50) : nullptr;
    for (int B : batches) {
      kv.batch = B;
      for (int tbl = 0; tbl < 2; ++tbl) {
        const int32_t* bt = tbl ? table : nullptr;
        for (int t = 1; t <= h.plan.max_tasks; t = t < 4 ? t + 1 : t * 2) {
          g.where = name + " cus " + std::to_string(cus) + " B " + std::to_string(B) + " tasks " + std::to_string(t) +
                    (packed ? " image" : "");
          const int st = t == 1 ? sp_probe_forward(&h, &kv, lens, bt, soft, &wt, logits, nullptr)
                                : sp_probe_forward_multi(&h, &kv, lens, bt, t, soft, &wt, logits, nullptr);
          g.expect(st == SP_OK, "forward status " + std::to_string(st));
        }
        g.where = name + " recursive cus " + std::to_string(cus) + " B " + std::to_string(B);
        for (int e3 = 0; e3 < 2; ++e3) {
          fu.w_hidden_fuse = e3 ? fake(33) : nullptr;
          const int st = sp_probe_forward_recursive(&h, &kv, lens, bt, soft, hidden, &fu, &wt, logits, nullptr);
          g.expect(st == SP_OK, "recursive status " + std::to_string(st));
        }
      }
    }
  }
  // host-checkable errors return before anything is enqueued
  g.where = name + " errors";
  kv.batch = cfg.max_batch + 1;
  g.expect(sp_probe_forward(&h, &kv, lens, nullptr, soft, &wt, logits, nullptr) == SP_ERR_CAPACITY, "capacity");
  kv.batch = 1;
  g.expect(sp_probe_forward(&h, &kv, lens, nullptr, (const char*)soft + 4, &wt, logits, nullptr) == SP_ERR_INVALID_ARG,
           "misaligned soft prompt");
  kv.block_size = 24;
  g.expect(sp_probe_forward(&h, &kv, lens, nullptr, soft, &wt, logits, nullptr) == SP_ERR_INVALID_ARG, "block size");
  kv.block_size = 16;
  g.expect(sp_probe_forward_multi(&h, &kv, lens, nullptr, h.plan.max_tasks + 1, soft, &wt, logits, nullptr) ==
               SP_ERR_INVALID_ARG, "task count");
  wt.packed = nullptr;
  wt.w_up = nullptr;
  g.expect(sp_probe_forward(&h, &kv, lens, nullptr, soft, &wt, logits, nullptr) == SP_ERR_INVALID_ARG, "null matrix");
  kv.batch = 0;
  g.expect(sp_probe_forward(&h, &kv, lens, nullptr, soft, &wt, logits, nullptr) == SP_OK, "empty batch");
  g.ws = nullptr;
}

}  // namespace

int main(int argc, char** argv) {
  const int n_random = argc > 1 ? std::atoi(argv[1]) : 300;
  const int cus_list[] = {80, 256, 304};
  struct Named { const char* name; sp_probe_config cfg; };
  const int LR = SP_FLAG_LAST_ROW_ONLY;
  const Named fixed[] = {
      {"tiny_f32", make_cfg(256, 4, 2, 64, 1024, 4, 2, SP_F32, SP_POOL_LAST, 4, 256, 0, 1, 0)},
      {"4b_bf16", make_cfg(2560, 32, 8, 128, 9728, 16, 2, SP_BF16, SP_POOL_LAST, 64, 4096, 0, 1, 0)},
      {"9b_bf16", make_cfg(4096, 32, 8, 128, 12288, 16, 3, SP_BF16, SP_POOL_LAST, 128, 8192, 0, 4, 0)},
      {"27b_bf16", make_cfg(5120, 40, 8, 128, 17408, 32, 2, SP_BF16, SP_POOL_LAST, 256, 32768, 0, 1, 0)},
      {"long_9b_bf16", make_cfg(4096, 32, 8, 128, 12288, 16, 4, SP_BF16, SP_POOL_LAST, 32, 131072, 0, 4, 0)},
      {"long_9b_bf16_lr", make_cfg(4096, 32, 8, 128, 12288, 16, 4, SP_BF16, SP_POOL_LAST, 32, 131072, LR, 4, 0)},
      {"small_g5_mean", make_cfg(640, 10, 2, 128, 1024, 8, 2, SP_BF16, SP_POOL_MEAN, 3, 1000, 0, 3, 0)},
      {"k64_tasks16", make_cfg(512, 8, 2, 128, 768, 64, 3, SP_BF16, SP_POOL_LAST, 5, 517, 0, 16, 0)},
      {"hd64_split", make_cfg(512, 8, 1, 64, 512, 17, 2, SP_BF16, SP_POOL_LAST, 7, 5000, 0, 2, 256)},
      {"f32_64rows", make_cfg(256, 16, 1, 64, 512, 4, 2, SP_F32, SP_POOL_MEAN, 3, 3000, 0, 1, 0)},
      {"empty_ctx", make_cfg(256, 4, 2, 128, 256, 1, 1, SP_BF16, SP_POOL_LAST, 2, 0, 0, 1, 0)},
  };
  for (const Named& n : fixed) {
    g.expect(check_config(&n.cfg) == SP_OK, std::string("config ") + n.name);
    for (int cus : cus_list) run_forwards(n.cfg, cus, n.name);
  }
  // seeded random shapes, valid and invalid: the checks must never misbehave,
  // and every accepted config must run its forwards inside the workspace
  std::mt19937_64 rng(20260601);
  auto pick = [&](std::initializer_list<int> v) { return *(v.begin() + rng() % v.size()); };
  int accepted = 0;
  for (int i = 0; i < n_random; ++i) {
    const int dtype = (int)(rng() % 2);
    const int hd = pick({64, 128, 96});
    const int nkv = pick({1, 2, 4, 8});
    const int G = pick({1, 2, 3, 4, 5, 8});
    const int d = (int)(32 * (1 + rng() % 64));
    const int I = (int)(32 * (1 + rng() % 96));
    const int k = (int)(1 + rng() % 64);
    const int C = (int)(1 + rng() % 8);
    const int B = (int)(1 + rng() % 40);
    const int N = (int)(rng() % 70000);
    const int tasks = (int)(rng() % 5);
    const int flags = (rng() % 3 == 0) ? LR : 0;
    const int pool = flags ? SP_POOL_LAST : (int)(rng() % 2);
    const int split = pick({0, 0, 256, 1024, 4096});
    const sp_probe_config cfg = make_cfg(d, nkv * G, nkv, hd, I, k, C, dtype, pool, B, N, flags, tasks, split);
    if (check_config(&cfg) != SP_OK) continue;
    ++accepted;
    run_forwards(cfg, cus_list[rng() % 3], "random " + std::to_string(i));
  }
  // configs the checks must refuse, including values that would overflow sizes
  const sp_probe_config bad[] = {
      make_cfg(16384, 4096, 1, 128, 1 << 20, 64, 64, SP_BF16, SP_POOL_LAST, 1 << 20, 1 << 30, 0, 64, 0),
      make_cfg(-32, 4, 2, 64, 64, 1, 1, SP_BF16, SP_POOL_LAST, 1, 1, 0, 1, 0),
      make_cfg(256, 4, 0, 64, 64, 1, 1, SP_BF16, SP_POOL_LAST, 1, 1, 0, 1, 0),
      make_cfg(256, 4, 2, 64, 64, 1, 1, SP_BF16, SP_POOL_LAST, 1, -5, 0, 1, 0),
      make_cfg(256, 4, 2, 64, 64, 1, 1, SP_BF16, SP_POOL_LAST, 1, 1, 0, 1, 384),
  };
  for (const sp_probe_config& c : bad) {
    g.where = "refused configs";
    g.expect(check_config(&c) != SP_OK, "accepted a bad config");
    g.expect(sp_probe_workspace_bytes(&c) == 0, "sized a bad config");
  }
  // host-only planning over compute-unit counts
  for (const Named& n : fixed)
    for (int cus = 1; cus <= 1024; cus = cus * 3 + 1) {
      int32_t sl = 0, ms = 0, rows = 0, grp = 0;
      size_t bytes = 0;
      g.where = std::string("plan ") + n.name;
      g.expect(sp_probe_plan_config(&n.cfg, cus, &sl, &ms, &rows, &grp, &bytes) == SP_OK, "plan status");
      g.expect(sl >= 256 && ms >= 1 && (int64_t)sl * ms >= n.cfg.max_seq_len && bytes > 0, "plan values");
    }
  // no device here: the device-facing calls report it and enqueue nothing
  {
    g.where = "no device";
    sp_probe_t* h = nullptr;
    g.expect(sp_probe_init(&fixed[1].cfg, &h) == SP_ERR_NO_DEVICE && h == nullptr, "init without a device");
    sp_kv_cache kv{};
    sp_probe_weights wt{};
    g.expect(sp_probe_forward_noalloc(&fixed[1].cfg, &kv, nullptr, nullptr, nullptr, &wt, nullptr, nullptr) ==
                 SP_ERR_NO_DEVICE, "forward without allocation, no device");
    g.expect(sp_probe_pack_weights(&fixed[1].cfg, &wt, nullptr, 0, nullptr) == SP_ERR_INVALID_ARG, "pack arguments");
  }
  std::printf("host runtime check: %ld checks, %d random configs accepted, %ld failures\n", g.checks, accepted,
              g.failures);
  return g.failures ? 1 : 0;
}
