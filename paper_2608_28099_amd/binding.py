"""ctypes binding of libsp_probe.so (include/sp_probe.h).

Argument marshalling only: every step of the forward runs in the library's HIP
kernels.  Loading fails loudly when the library has not been built.  torch is
used for device buffers and the current stream.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libsp_probe.so")

SP_OK = 0
STATUS = {0: "SP_OK", -1: "SP_ERR_INVALID_ARG", -2: "SP_ERR_UNSUPPORTED", -3: "SP_ERR_NO_DEVICE",
          -4: "SP_ERR_OUT_OF_MEMORY", -5: "SP_ERR_HIP", -6: "SP_ERR_CAPACITY",
          -7: "SP_ERR_DEVICE_DATA", -8: "SP_ERR_RANGE", -9: "SP_ERR_INTERNAL"}
SP_ERR_DEVICE_DATA, SP_ERR_RANGE, SP_ERR_INTERNAL = -7, -8, -9
SP_F32, SP_BF16 = 0, 1
SP_POOL_LAST, SP_POOL_MEAN = 0, 1
SP_FLAG_DEBUG, SP_FLAG_PROFILE, SP_FLAG_LAST_ROW_ONLY = 1, 2, 4
SP_TAP_QKV, SP_TAP_ATTN, SP_TAP_A, SP_TAP_Y, SP_TAP_X = 0, 1, 2, 3, 4
SP_N_STAGES = 8
STAGES = ("soft_prep", "attention", "merge", "o_proj", "post_norm", "gate_up", "down", "classifier")

# Every function the header declares, with its C signature.
EXPORTS = ("sp_probe_workspace_bytes", "sp_probe_init", "sp_probe_forward",
           "sp_probe_forward_multi", "sp_probe_forward_recursive", "sp_probe_destroy", "sp_probe_status_string",
           "sp_probe_tap_bytes", "sp_probe_copy_tap", "sp_probe_check_device_error",
           "sp_probe_profile_read", "sp_probe_plan", "sp_probe_plan_recursive", "sp_probe_plan_config",
           "sp_probe_packed_bytes", "sp_probe_pack_weights", "sp_probe_measure_read", "sp_probe_measure_mfma",
           "sp_probe_forward_noalloc")


class sp_probe_config(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("intermediate", ctypes.c_int32), ("k", ctypes.c_int32),
                ("n_classes", ctypes.c_int32), ("dtype", ctypes.c_int32), ("pool", ctypes.c_int32),
                ("rms_eps", ctypes.c_float), ("rope_base", ctypes.c_double),
                ("max_batch", ctypes.c_int32), ("max_seq_len", ctypes.c_int32),
                ("split_len", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("max_tasks", ctypes.c_int32)]


class sp_kv_cache(ctypes.Structure):
    _fields_ = [("k_base", ctypes.c_void_p), ("v_base", ctypes.c_void_p),
                ("num_blocks", ctypes.c_int64),
                ("k_stride_block", ctypes.c_int64), ("k_stride_head", ctypes.c_int64),
                ("v_stride_block", ctypes.c_int64), ("v_stride_head", ctypes.c_int64),
                ("block_size", ctypes.c_int32), ("max_blocks_per_seq", ctypes.c_int32),
                ("batch", ctypes.c_int32)]


class sp_probe_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("in_norm", "w_q", "w_k", "w_v", "w_o", "post_norm", "w_gate", "w_up", "w_down",
                 "final_norm", "w_cls", "b_cls", "cls_rows")] + [("cls_vocab", ctypes.c_int64),
                                                                  ("packed", ctypes.c_void_p)]



class sp_probe_fusion(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("fc_norm_hidden", "fc_norm_embed", "w_fc", "w_hidden_fuse")]


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the library (once).  Raises if it is missing: there is no fallback."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() "
                           "(there is no non-HIP fallback)")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    vp = ctypes.c_void_p
    lib.sp_probe_workspace_bytes.argtypes = [P(sp_probe_config)]
    lib.sp_probe_workspace_bytes.restype = ctypes.c_size_t
    lib.sp_probe_init.argtypes = [P(sp_probe_config), P(vp)]
    lib.sp_probe_init.restype = ctypes.c_int
    lib.sp_probe_forward.argtypes = [vp, P(sp_kv_cache), vp, vp, vp, P(sp_probe_weights), vp, vp]
    lib.sp_probe_forward.restype = ctypes.c_int
    lib.sp_probe_forward_noalloc.argtypes = [P(sp_probe_config), P(sp_kv_cache), vp, vp, vp, P(sp_probe_weights),
                                             vp, vp]
    lib.sp_probe_forward_noalloc.restype = ctypes.c_int
    lib.sp_probe_forward_multi.argtypes = [vp, P(sp_kv_cache), vp, vp, ctypes.c_int32, vp,
                                           P(sp_probe_weights), vp, vp]
    lib.sp_probe_forward_multi.restype = ctypes.c_int
    lib.sp_probe_forward_recursive.argtypes = [vp, P(sp_kv_cache), vp, vp, vp, vp, P(sp_probe_fusion),
                                               P(sp_probe_weights), vp, vp]
    lib.sp_probe_forward_recursive.restype = ctypes.c_int
    lib.sp_probe_destroy.argtypes = [vp]
    lib.sp_probe_destroy.restype = ctypes.c_int
    lib.sp_probe_status_string.argtypes = [ctypes.c_int]
    lib.sp_probe_status_string.restype = ctypes.c_char_p
    lib.sp_probe_tap_bytes.argtypes = [vp, ctypes.c_int, ctypes.c_int32]
    lib.sp_probe_tap_bytes.restype = ctypes.c_size_t
    lib.sp_probe_copy_tap.argtypes = [vp, ctypes.c_int, ctypes.c_int32, vp, ctypes.c_size_t, vp]
    lib.sp_probe_copy_tap.restype = ctypes.c_int
    lib.sp_probe_check_device_error.argtypes = [vp, vp]
    lib.sp_probe_check_device_error.restype = ctypes.c_int
    lib.sp_probe_profile_read.argtypes = [vp, P(ctypes.c_float), ctypes.c_int32, P(ctypes.c_int32)]
    lib.sp_probe_profile_read.restype = ctypes.c_int
    lib.sp_probe_plan.argtypes = [vp, ctypes.c_int32] + [P(ctypes.c_int32)] * 4
    lib.sp_probe_plan.restype = ctypes.c_int
    lib.sp_probe_plan_recursive.argtypes = [vp, ctypes.c_int32] + [P(ctypes.c_int32)] * 4
    lib.sp_probe_plan_recursive.restype = ctypes.c_int
    lib.sp_probe_plan_config.argtypes = [P(sp_probe_config), ctypes.c_int32] + [P(ctypes.c_int32)] * 4 + \
        [P(ctypes.c_size_t)]
    lib.sp_probe_plan_config.restype = ctypes.c_int
    lib.sp_probe_packed_bytes.argtypes = [P(sp_probe_config)]
    lib.sp_probe_packed_bytes.restype = ctypes.c_size_t
    lib.sp_probe_pack_weights.argtypes = [P(sp_probe_config), P(sp_probe_weights), vp, ctypes.c_size_t, vp]
    lib.sp_probe_pack_weights.restype = ctypes.c_int
    lib.sp_probe_measure_read.argtypes = [vp, ctypes.c_size_t, ctypes.c_int32, vp, P(ctypes.c_float), vp]
    lib.sp_probe_measure_read.restype = ctypes.c_int
    lib.sp_probe_measure_mfma.argtypes = [ctypes.c_int32, vp, P(ctypes.c_float), vp]
    lib.sp_probe_measure_mfma.restype = ctypes.c_int
    _lib = lib
    return lib


class ProbeError(RuntimeError):
    def __init__(self, status: int, what: str = ""):
        self.status = status
        super().__init__(f"{what}: {STATUS.get(status, status)}")


def _check(status: int, what: str) -> None:
    if status != SP_OK:
        raise ProbeError(status, what)


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


# ---------------------------------------------------------------- thin wrappers (C names)

def sp_probe_workspace_bytes(cfg: sp_probe_config) -> int:
    return load().sp_probe_workspace_bytes(ctypes.byref(cfg))


def sp_probe_init(cfg: sp_probe_config) -> int:
    h = ctypes.c_void_p()
    _check(load().sp_probe_init(ctypes.byref(cfg), ctypes.byref(h)), "sp_probe_init")
    return h.value


def sp_probe_forward(h, kv: sp_kv_cache, seq_lens, block_table, soft_prompt,
                     weights: sp_probe_weights, logits, stream) -> int:
    return load().sp_probe_forward(h, ctypes.byref(kv), seq_lens, block_table, soft_prompt,
                                   ctypes.byref(weights), logits, stream)


def sp_probe_forward_noalloc(cfg: sp_probe_config, kv: sp_kv_cache, seq_lens, block_table, soft_prompt,
                             weights: sp_probe_weights, logits, stream) -> int:
    return load().sp_probe_forward_noalloc(ctypes.byref(cfg), ctypes.byref(kv), seq_lens, block_table, soft_prompt,
                                           ctypes.byref(weights), logits, stream)


def sp_probe_forward_multi(h, kv: sp_kv_cache, seq_lens, block_table, n_tasks: int, soft_prompts,
                           weights: sp_probe_weights, logits, stream) -> int:
    return load().sp_probe_forward_multi(h, ctypes.byref(kv), seq_lens, block_table, n_tasks,
                                         soft_prompts, ctypes.byref(weights), logits, stream)


def sp_probe_forward_recursive(h, kv: sp_kv_cache, seq_lens, block_table, soft_prompt, hidden_last,
                               fusion: sp_probe_fusion, weights: sp_probe_weights, logits, stream) -> int:
    return load().sp_probe_forward_recursive(h, ctypes.byref(kv), seq_lens, block_table, soft_prompt,
                                             hidden_last, ctypes.byref(fusion), ctypes.byref(weights),
                                             logits, stream)


def sp_probe_destroy(h) -> int:
    return load().sp_probe_destroy(h)


def sp_probe_status_string(status: int) -> str:
    return load().sp_probe_status_string(status).decode()


def sp_probe_plan_config(cfg: sp_probe_config, num_cus: int):
    """Host-only split plan and workspace size of cfg on a device of num_cus compute units."""
    vals = [ctypes.c_int32() for _ in range(4)]
    ws = ctypes.c_size_t()
    st = load().sp_probe_plan_config(ctypes.byref(cfg), num_cus, *[ctypes.byref(v) for v in vals],
                                     ctypes.byref(ws))
    _check(st, "sp_probe_plan_config")
    return {"split_len": vals[0].value, "max_splits": vals[1].value, "rows_per_kv_head": vals[2].value,
            "query_groups": vals[3].value, "workspace_bytes": ws.value}


def measure_read_gbps(buf, reps: int = 10, stream=None) -> float:
    """Streaming-read rate of the device over the device tensor buf (GB/s)."""
    import torch
    sink = torch.zeros(4, dtype=torch.int32, device=buf.device)
    if stream is None:
        stream = torch.cuda.current_stream(buf.device).cuda_stream
    out = ctypes.c_float()
    _check(load().sp_probe_measure_read(buf.data_ptr(), buf.numel() * buf.element_size(), reps, sink.data_ptr(),
                                        ctypes.byref(out), stream), "sp_probe_measure_read")
    return float(out.value)


def measure_mfma_tflops(device, iters: int = 20000, stream=None) -> float:
    """Sustained dense fp16 matrix-core rate of the device (TFLOP/s)."""
    import torch
    sink = torch.zeros(4, dtype=torch.int32, device=device)
    if stream is None:
        stream = torch.cuda.current_stream(device).cuda_stream
    out = ctypes.c_float()
    _check(load().sp_probe_measure_mfma(iters, sink.data_ptr(), ctypes.byref(out), stream), "sp_probe_measure_mfma")
    return float(out.value)


def sp_probe_packed_bytes(cfg: sp_probe_config) -> int:
    return load().sp_probe_packed_bytes(ctypes.byref(cfg))


def sp_probe_pack_weights(cfg: sp_probe_config, weights: sp_probe_weights, packed, packed_bytes: int,
                          stream) -> int:
    return load().sp_probe_pack_weights(ctypes.byref(cfg), ctypes.byref(weights), packed, packed_bytes, stream)


# ---------------------------------------------------------------- torch-facing helpers

def make_config(w, max_batch: Optional[int] = None, max_seq_len: Optional[int] = None,
                split_len: int = 0, flags: int = 0, max_tasks: int = 1) -> sp_probe_config:
    """sp_probe_config for a paper_2608_28099_amd.configs.Workload."""
    return sp_probe_config(
        hidden=w.hidden, n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim,
        intermediate=w.intermediate, k=w.k, n_classes=w.n_classes,
        dtype=SP_BF16 if w.dtype == "bf16" else SP_F32,
        pool=SP_POOL_MEAN if w.pool == "mean" else SP_POOL_LAST,
        rms_eps=w.rms_eps, rope_base=w.rope_base,
        max_batch=max_batch if max_batch is not None else w.batch,
        max_seq_len=max_seq_len if max_seq_len is not None else w.max_seq_len(),
        split_len=split_len, flags=flags, max_tasks=max_tasks)


def make_kv(kv, batch: Optional[int] = None) -> sp_kv_cache:
    """sp_kv_cache for a paper_2608_28099_amd.inputs.KVCache (one pool tensor)."""
    base = kv.pool.data_ptr()
    esz = kv.pool.element_size()
    return sp_kv_cache(
        k_base=base, v_base=base + kv.v_offset * esz, num_blocks=kv.num_blocks,
        k_stride_block=kv.stride_block, k_stride_head=kv.stride_head,
        v_stride_block=kv.stride_block, v_stride_head=kv.stride_head,
        block_size=kv.block_size, max_blocks_per_seq=kv.max_blocks_per_seq,
        batch=kv.seq_lens.shape[0] if batch is None else batch)


def make_weights(params: dict) -> sp_probe_weights:
    """params: the head's tensors; optional cls_rows (device int32) selects rows of
    w_cls, a vocabulary matrix of cls_vocab rows (default: its first dimension);
    optional packed: a uint8 tensor holding the fp16 weight image (pack_weights)."""
    wt = sp_probe_weights(**{n: _ptr(params.get(n)) for n in
                             ("in_norm", "w_q", "w_k", "w_v", "w_o", "post_norm", "w_gate",
                              "w_up", "w_down", "final_norm", "w_cls", "b_cls", "cls_rows", "packed")})
    if params.get("cls_rows") is not None:
        wt.cls_vocab = params.get("cls_vocab", params["w_cls"].shape[0])
    return wt


def make_fusion(fusion: dict) -> sp_probe_fusion:
    return sp_probe_fusion(**{n: _ptr(fusion.get(n)) for n in
                              ("fc_norm_hidden", "fc_norm_embed", "w_fc", "w_hidden_fuse")})


def pack_weights(w, params: dict, stream=None, max_tasks: int = 1):
    """The fp16 weight image of the head in params (a device uint8 tensor), made by
    sp_probe_pack_weights; pass it as params["packed"]."""
    import torch
    cfg = make_config(w, max_tasks=max_tasks)
    n = sp_probe_packed_bytes(cfg)
    if n == 0:
        raise ProbeError(-2, "sp_probe_packed_bytes")
    dev = params["w_q"].device
    img = torch.empty(n, dtype=torch.uint8, device=dev)
    if stream is None:
        stream = torch.cuda.current_stream(dev).cuda_stream
    _check(sp_probe_pack_weights(cfg, make_weights(params), img.data_ptr(), n, stream), "sp_probe_pack_weights")
    return img


class Probe:
    """One library handle (workspace) for a workload shape."""

    def __init__(self, w, max_batch=None, max_seq_len=None, split_len=0, flags=0, max_tasks=1):
        self.w = w
        self.cfg = make_config(w, max_batch, max_seq_len, split_len, flags, max_tasks)
        self.h = sp_probe_init(self.cfg)
        self.lib = load()

    def close(self):
        if self.h:
            _check(sp_probe_destroy(self.h), "sp_probe_destroy")
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def forward(self, kv, params: dict, logits=None, stream=None, batch=None):
        import torch
        B = kv.seq_lens.shape[0] if batch is None else batch
        if logits is None:
            logits = torch.empty((B, self.w.n_classes), dtype=torch.float32, device=kv.pool.device)
        if stream is None:
            stream = torch.cuda.current_stream(kv.pool.device).cuda_stream
        self._kv = make_kv(kv, B)
        self._wt = make_weights(params)
        st = sp_probe_forward(self.h, self._kv, kv.seq_lens.data_ptr(), _ptr(kv.block_table),
                              params["soft_prompt"].data_ptr(), self._wt, logits.data_ptr(), stream)
        _check(st, "sp_probe_forward")
        return logits

    def forward_multi(self, kv, params: dict, soft_prompts, w_cls, b_cls=None, logits=None,
                      stream=None, batch=None, cls_rows=None):
        """T tasks in one call: soft_prompts [T][k][d], w_cls [T][C][d], b_cls [T][C] or
        None (the rest of params is the shared head); returns logits [B][T][C]."""
        import torch
        B = kv.seq_lens.shape[0] if batch is None else batch
        T = soft_prompts.shape[0]
        if logits is None:
            logits = torch.empty((B, T, self.w.n_classes), dtype=torch.float32, device=kv.pool.device)
        if stream is None:
            stream = torch.cuda.current_stream(kv.pool.device).cuda_stream
        self._kv = make_kv(kv, B)
        self._wt = make_weights(dict(params, w_cls=w_cls, b_cls=b_cls, cls_rows=cls_rows))
        st = sp_probe_forward_multi(self.h, self._kv, kv.seq_lens.data_ptr(), _ptr(kv.block_table), T,
                                    soft_prompts.data_ptr(), self._wt, logits.data_ptr(), stream)
        _check(st, "sp_probe_forward_multi")
        return logits

    def forward_recursive(self, kv, params: dict, fusion: dict, logits=None, stream=None, batch=None):
        """Recursive SP-k; fusion holds fc_norm_hidden, fc_norm_embed, w_fc and
        hidden_last [B][d] (paper_2608_28099_amd.inputs.fusion_params)."""
        import torch
        B = kv.seq_lens.shape[0] if batch is None else batch
        if logits is None:
            logits = torch.empty((B, self.w.n_classes), dtype=torch.float32, device=kv.pool.device)
        if stream is None:
            stream = torch.cuda.current_stream(kv.pool.device).cuda_stream
        self._kv = make_kv(kv, B)
        self._wt = make_weights(params)
        self._fu = make_fusion(fusion)
        st = sp_probe_forward_recursive(self.h, self._kv, kv.seq_lens.data_ptr(), _ptr(kv.block_table),
                                        params["soft_prompt"].data_ptr(), _ptr(fusion["hidden_last"]),
                                        self._fu, self._wt, logits.data_ptr(), stream)
        _check(st, "sp_probe_forward_recursive")
        return logits

    def tap(self, tap: int, batch: int, device):
        import torch
        n = self.lib.sp_probe_tap_bytes(self.h, tap, batch)
        buf = torch.empty(n, dtype=torch.uint8, device=device)
        stream = torch.cuda.current_stream(device).cuda_stream
        _check(self.lib.sp_probe_copy_tap(self.h, tap, batch, buf.data_ptr(), n, stream), "copy_tap")
        return buf

    def plan(self, batch: int):
        vals = [ctypes.c_int32() for _ in range(4)]
        _check(self.lib.sp_probe_plan(self.h, batch, *[ctypes.byref(v) for v in vals]), "plan")
        return {"split_len": vals[0].value, "max_splits": vals[1].value,
                "rows_per_kv_head": vals[2].value, "query_groups": vals[3].value}

    def plan_recursive(self, batch: int):
        vals = [ctypes.c_int32() for _ in range(4)]
        _check(self.lib.sp_probe_plan_recursive(self.h, batch, *[ctypes.byref(v) for v in vals]),
               "plan_recursive")
        return {"split_len": vals[0].value, "max_splits": vals[1].value,
                "rows_per_kv_head": vals[2].value, "query_groups": vals[3].value}

    def check_device_error(self, stream=None) -> int:
        import torch
        if stream is None:
            stream = torch.cuda.current_stream().cuda_stream
        return self.lib.sp_probe_check_device_error(self.h, stream)

    def profile_read(self):
        arr = (ctypes.c_float * SP_N_STAGES)()
        n = ctypes.c_int32()
        _check(self.lib.sp_probe_profile_read(self.h, arr, SP_N_STAGES, ctypes.byref(n)), "profile")
        return dict(zip(STAGES, list(arr))), n.value
