"""ctypes binding of include/darts.h.  Argument marshalling only: every step of
the rollout runs in the HIP library (libdarts.so, built for gfx950).  PyTorch
provides device memory and the stream; there is no CPU fallback -- a missing
library raises."""
import ctypes as C
import os

import numpy as np

DARTS_OK, DARTS_EINVAL, DARTS_ENOMEM, DARTS_ESTATE, DARTS_EHIP = 0, 1, 2, 3, 4
DARTS_F32, DARTS_BF16 = 0, 1
FLAG_NO_ABORT, FLAG_PERMUTE_PAGES, FLAG_TIMING, FLAG_SHARED_PREFIX, FLAG_STEP_TIMES = 0x1, 0x2, 0x4, 0x8, 0x10
FLAG_STREAM = 0x20

_HERE = os.path.dirname(os.path.abspath(__file__))
lib_path = os.path.join(_HERE, "libdarts.so")


class DartsError(RuntimeError):
    def __init__(self, status, msg=""):
        super().__init__(f"darts status {status}: {msg}")
        self.status = status


class ModelCfg(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn_dim", C.c_int32),
                ("vocab", C.c_int32), ("n_experts", C.c_int32), ("top_k", C.c_int32),
                ("expert_ffn", C.c_int32), ("rope_theta", C.c_float), ("rms_eps", C.c_float),
                ("dtype", C.c_int32), ("weight_seed", C.c_uint64), ("weights", C.c_void_p)]


class RunCfg(C.Structure):
    _fields_ = [("n_prompts", C.c_int32), ("prompt_len", C.c_int32), ("cap", C.c_int32),
                ("L", C.c_int32), ("m_up", C.c_int32), ("page_size", C.c_int32),
                ("kv_pool_bytes", C.c_uint64), ("sample_seed", C.c_uint64),
                ("temperature", C.c_float), ("flags", C.c_uint32),
                ("page_perm_seed", C.c_uint64), ("stream", C.c_void_p), ("traj_base", C.c_int32)]


class StepOut(C.Structure):
    _fields_ = [("traj_id", C.c_void_p), ("token", C.c_void_p), ("sampled", C.c_void_p),
                ("logprob", C.c_void_p), ("entropy", C.c_void_p), ("finished", C.c_void_p),
                ("n_rows", C.c_int32)]


class Stats(C.Structure):
    _fields_ = [("steps", C.c_int64), ("tokens_decoded", C.c_int64), ("n_pages", C.c_int64),
                ("pages_used", C.c_int64), ("pages_hwm", C.c_int64), ("n_live", C.c_int32),
                ("n_done", C.c_int32), ("attn_ms", C.c_double), ("attn_bytes", C.c_double),
                ("attn_launches", C.c_int64), ("gemm_ms", C.c_double), ("gemm_flop", C.c_double),
                ("gemm_launches", C.c_int64), ("gemm_cls_ms", C.c_double * 6),
                ("gemm_cls_flop", C.c_double * 6), ("attn_traj_bytes", C.c_double),
                ("moe_expert_ms", C.c_double * 2), ("moe_expert_bytes", C.c_double * 2),
                ("moe_expert_launches", C.c_int64 * 2)]


_P = C.c_void_p
_SIGS = {
    "darts_init": (C.c_int, [C.POINTER(ModelCfg), C.c_int32, C.c_int32, C.POINTER(RunCfg), C.POINTER(_P)]),
    "darts_prefill": (C.c_int, [_P, _P, _P, _P, C.POINTER(StepOut)]),
    "darts_decode_step": (C.c_int, [_P, _P, C.POINTER(StepOut)]),
    "darts_select_and_prune": (C.c_int, [_P, _P, _P, C.POINTER(C.c_int32), C.POINTER(C.c_int32)]),
    "darts_get_stats": (C.c_int, [_P, C.POINTER(Stats)]),
    "darts_get_traj_scores": (C.c_int, [_P, _P, _P, _P, _P]),
    "darts_debug_logits": (C.c_int, [_P, _P, C.POINTER(C.c_int32)]),
    "darts_destroy": (C.c_int, [_P]),
    "darts_weight_count": (C.c_int32, [C.POINTER(ModelCfg)]),
    "darts_debug_moe_routing": (C.c_int, [_P, _P, _P, _P, C.c_int64]),
    "darts_debug_fill_kv": (C.c_int, [_P, C.c_int32]),
    "darts_reset": (C.c_int, [_P]),
    "darts_set_plan": (C.c_int, [_P, _P]),
    "darts_prompt_length_std": (C.c_int, [_P, _P, C.c_int32, C.c_int32, _P]),
    "darts_ema_update": (C.c_int, [_P, _P, _P, C.c_int32, C.c_double]),
    "darts_redundancy_budget": (C.c_int, [C.c_double, C.c_double, C.c_double, C.c_int32, C.c_int32,
                                          C.POINTER(C.c_int64)]),
    "darts_allocate_redundancy": (C.c_int, [_P, _P, C.c_int32, C.c_int32, C.c_int32, C.c_int64, _P]),
    "darts_get_step_times": (C.c_int, [_P, _P, _P, C.c_int32, C.POINTER(C.c_int32), C.POINTER(C.c_float)]),
    "darts_rollout_cost": (C.c_int, [_P, C.c_int32, _P, C.POINTER(C.c_double)]),
    "darts_rollout_cost_dp": (C.c_int, [_P, _P, C.c_int32, C.c_int32, _P, C.POINTER(C.c_double)]),
    "darts_fit_ptl": (C.c_int, [_P, _P, C.c_int32, _P]),
    "darts_stream_chunks": (C.c_int, [_P, C.c_int64, C.c_int32, _P, _P, _P, C.c_int64,
                                      C.POINTER(C.c_int32), C.POINTER(C.c_int64)]),
    "darts_group_advantages": (C.c_int, [_P, C.c_int32, C.c_int32, _P, C.c_int32, C.c_float, _P, _P]),
    "darts_strerror": (C.c_char_p, [C.c_int]),
    "darts_last_error": (C.c_char_p, [_P]),
    "darts_fill_uniform": (C.c_int, [_P, C.c_uint64, C.c_int32, C.c_uint64, C.c_int32, _P]),
    "darts_fill_kv_pool": (C.c_int, [_P, _P, C.c_int64, C.c_int32, C.c_int32, C.c_uint64, C.c_int32, _P]),
    "darts_attn_workspace_bytes": (C.c_size_t, [C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32]),
    "darts_attn_decode": (C.c_int, [_P, _P, _P, C.c_int64, _P, C.c_int32, _P, C.c_int32, C.c_int32,
                                    C.c_int32, C.c_int32, C.c_int32, C.c_int32, _P, _P, C.c_size_t, _P]),
    "darts_attn_decode_noalloc": (C.c_int, [_P, _P, _P, C.c_int64, _P, C.c_int32, _P, C.c_int32,
                                            C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32, _P, _P]),
    "darts_attn_shared_workspace_bytes": (C.c_size_t, [C.c_int32] * 6),
    "darts_attn_decode_shared": (C.c_int, [_P, _P, _P, C.c_int64, _P, C.c_int32, C.c_int32, _P,
                                           C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                           C.c_int32, C.c_int32, C.c_int32, _P, _P, C.c_size_t, _P]),
    "darts_sample": (C.c_int, [_P, C.c_int32, C.c_int32, C.c_int32, C.c_uint64, _P, _P, C.c_float,
                               _P, _P, _P, _P, _P]),
    "darts_debug_gumbel": (C.c_int, [_P, _P, C.c_int64, _P]),
    "darts_debug_gumbel_fast": (C.c_int, [_P, _P, C.c_int64, _P]),
    "darts_stream_read": (C.c_int, [_P, C.c_int64, _P, _P]),
    "darts_sampler_gumbel_bound": (C.c_float, []),
    "darts_gemm_workspace_bytes": (C.c_size_t, [C.c_int32, C.c_int32, C.c_int32]),
    "darts_gemm": (C.c_int, [_P, _P, _P, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                             _P, C.c_size_t, _P]),
    "darts_select_groups": (C.c_int, [_P, _P, _P, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                      C.c_int32, C.c_int32, _P, _P, _P, _P, _P, _P, _P, _P]),
}

_lib = None


def load_library(path=None):
    """Load libdarts.so (raises if it is missing: there is no fallback path)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or lib_path
    if not os.path.exists(p):
        raise DartsError(DARTS_EHIP, f"HIP library not built: {p} (run __graft_entry__.build())")
    lib = C.CDLL(p)
    for name, (res, args) in _SIGS.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    if path is None:
        _lib = lib
    return lib


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def _check(status, ctx=None):
    if status != DARTS_OK:
        lib = load_library()
        msg = lib.darts_strerror(status).decode()
        if ctx:
            extra = lib.darts_last_error(ctx).decode()
            if extra:
                msg += " | " + extra
        raise DartsError(status, msg)


# ---------------------------------------------------------------- stateless
def darts_fill_uniform(dst, tensor_id, seed, dtype, stream=None):
    _check(load_library().darts_fill_uniform(_ptr(dst), dst.numel(), tensor_id, seed, dtype,
                                             _stream(stream)))


def darts_fill_kv_pool(k_pool, v_pool, n_pages, n_kv_heads, head_dim, seed, dtype, stream=None):
    _check(load_library().darts_fill_kv_pool(_ptr(k_pool), _ptr(v_pool), n_pages, n_kv_heads,
                                             head_dim, seed, dtype, _stream(stream)))


def darts_attn_workspace_bytes(n_rows, n_q_heads, n_kv_heads, head_dim, max_ctx):
    return int(load_library().darts_attn_workspace_bytes(n_rows, n_q_heads, n_kv_heads, head_dim,
                                                         max_ctx))


def darts_attn_decode(q, k_pool, v_pool, n_pages, page_table, ctx_len, n_q_heads, n_kv_heads,
                      head_dim, max_ctx, dtype, out, workspace, stream=None, n_rows=None):
    """ctx_len None: every one of n_rows rows has max_ctx keys."""
    if ctx_len is not None:
        n_rows = ctx_len.numel()
    elif n_rows is None:
        raise ValueError("n_rows is required when ctx_len is None")
    _check(load_library().darts_attn_decode(
        _ptr(q), _ptr(k_pool), _ptr(v_pool), n_pages, _ptr(page_table), page_table.shape[1],
        _ptr(ctx_len), n_rows, n_q_heads, n_kv_heads, head_dim, max_ctx, dtype, _ptr(out),
        _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(stream)))


ATTN_NOALLOC_SCRATCH_BYTES = 64 << 20


def darts_attn_decode_noalloc(q, k_pool, v_pool, n_pages, page_table, ctx_len, n_q_heads, n_kv_heads,
                              head_dim, max_ctx, dtype, out, stream=None, n_rows=None):
    """darts_attn_decode with the library's own workspace array (no allocation)."""
    if ctx_len is not None:
        n_rows = ctx_len.numel()
    elif n_rows is None:
        raise ValueError("n_rows is required when ctx_len is None")
    _check(load_library().darts_attn_decode_noalloc(
        _ptr(q), _ptr(k_pool), _ptr(v_pool), n_pages, _ptr(page_table), page_table.shape[1],
        _ptr(ctx_len), n_rows, n_q_heads, n_kv_heads, head_dim, max_ctx, dtype, _ptr(out),
        _stream(stream)))


def darts_attn_shared_workspace_bytes(n_rows, n_q_heads, n_kv_heads, head_dim, ctx_len, prefix_pages):
    return int(load_library().darts_attn_shared_workspace_bytes(n_rows, n_q_heads, n_kv_heads,
                                                                head_dim, ctx_len, prefix_pages))


def darts_attn_decode_shared(q, k_pool, v_pool, n_pages, page_table, row_traj, m, prefix_pages,
                             ctx_len, n_q_heads, n_kv_heads, head_dim, dtype, out, workspace,
                             stream=None):
    n_rows = row_traj.numel()
    _check(load_library().darts_attn_decode_shared(
        _ptr(q), _ptr(k_pool), _ptr(v_pool), n_pages, _ptr(page_table), page_table.shape[1],
        page_table.shape[0], _ptr(row_traj), m, prefix_pages, ctx_len, n_rows, n_q_heads, n_kv_heads,
        head_dim, dtype, _ptr(out), _ptr(workspace), workspace.numel() * workspace.element_size(),
        _stream(stream)))


def darts_sample(logits, dtype, seed, traj, step, temperature, force, token, logprob, entropy,
                 stream=None):
    n_rows, vocab = logits.shape
    _check(load_library().darts_sample(_ptr(logits), n_rows, vocab, dtype, seed, _ptr(traj),
                                       _ptr(step), float(temperature), _ptr(force), _ptr(token),
                                       _ptr(logprob), _ptr(entropy), _stream(stream)))


def darts_select_groups(status, length, mean_lp, m, k, L, m_up, early_stop, kept, complete,
                        page_off=None, pages=None, free_out=None, n_free=None, work=None, stream=None):
    """Stateless Alg. 2 over groups of m; with page lists (CSR page_off / pages)
    the completed groups' pages go to free_out and their count to n_free."""
    _check(load_library().darts_select_groups(_ptr(status), _ptr(length), _ptr(mean_lp),
                                              status.numel(), m, k, L, m_up, early_stop, _ptr(kept),
                                              _ptr(complete), _ptr(page_off), _ptr(pages), _ptr(free_out),
                                              _ptr(n_free), _ptr(work), _stream(stream)))


def darts_group_advantages(kept, reward, adv, eps=1e-6, stream=None):
    """kept: int32 [n_groups, k] device tensor; reward: float32 [n_traj]; adv: like kept, float32."""
    n_groups, k = kept.shape
    _check(load_library().darts_group_advantages(_ptr(kept), n_groups, k, _ptr(reward), reward.numel(),
                                                 eps, _ptr(adv), _stream(stream)))


def darts_gemm_workspace_bytes(M, N, K):
    return int(load_library().darts_gemm_workspace_bytes(M, N, K))


def darts_gemm(a, w, c, M, N, K, dtype, epilogue, workspace=None, stream=None):
    wb = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(load_library().darts_gemm(_ptr(a), _ptr(w), _ptr(c), M, N, K, dtype, epilogue,
                                     _ptr(workspace), wb, _stream(stream)))


def darts_debug_gumbel(u, g, stream=None):
    _check(load_library().darts_debug_gumbel(_ptr(u), _ptr(g), u.numel(), _stream(stream)))


def darts_debug_gumbel_fast(u, g, stream=None):
    _check(load_library().darts_debug_gumbel_fast(_ptr(u), _ptr(g), u.numel(), _stream(stream)))


def darts_stream_read(src, sink, stream=None):
    _check(load_library().darts_stream_read(_ptr(src), src.numel() * src.element_size(), _ptr(sink),
                                            _stream(stream)))


def darts_sampler_gumbel_bound():
    return float(load_library().darts_sampler_gumbel_bound())


# ---------------------------------------------------------------- planning
def _np_ptr(a):
    return None if a is None else C.c_void_p(a.ctypes.data)


def darts_prompt_length_std(lengths, plan, n_prompts, m):
    """lengths: int32 [n_prompts*m] host array; plan: None or int32 [n_prompts]."""
    import numpy as np
    ln = np.ascontiguousarray(lengths, dtype=np.int32)
    pl = None if plan is None else np.ascontiguousarray(plan, dtype=np.int32)
    out = np.zeros(n_prompts, dtype=np.float64)
    _check(load_library().darts_prompt_length_std(_np_ptr(ln), _np_ptr(pl), n_prompts, m, _np_ptr(out)))
    return out


def darts_ema_update(est, seen, obs, alpha=0.5):
    """In place on float64 `est` and uint8 `seen`; NaN in `obs` = not observed."""
    import numpy as np
    assert est.dtype == np.float64 and seen.dtype == np.uint8 and est.flags.c_contiguous
    o = np.ascontiguousarray(obs, dtype=np.float64)
    _check(load_library().darts_ema_update(_np_ptr(est), _np_ptr(seen), _np_ptr(o), len(est), alpha))


def darts_redundancy_budget(rho, lam, k_cost, n_prompts, M):
    out = C.c_int64()
    _check(load_library().darts_redundancy_budget(rho, lam, k_cost, n_prompts, M, C.byref(out)))
    return out.value


def darts_allocate_redundancy(sigma, m_low, m_up, m_total, seen=None):
    import numpy as np
    sg = np.ascontiguousarray(sigma, dtype=np.float64)
    sn = None if seen is None else np.ascontiguousarray(seen, dtype=np.uint8)
    out = np.zeros(len(sg), dtype=np.int32)
    _check(load_library().darts_allocate_redundancy(_np_ptr(sg), _np_ptr(sn), len(sg), m_low, m_up,
                                                    m_total, _np_ptr(out)))
    return out


def darts_rollout_cost(lengths, ptl):
    import numpy as np
    ln = np.ascontiguousarray(lengths, dtype=np.int32)
    p = np.ascontiguousarray(ptl, dtype=np.float64)
    out = C.c_double()
    _check(load_library().darts_rollout_cost(_np_ptr(ln), len(ln), _np_ptr(p), C.byref(out)))
    return out.value


def darts_rollout_cost_dp(lengths, ranks, n_ranks, ptl):
    import numpy as np
    ln = np.ascontiguousarray(lengths, dtype=np.int32)
    rk = np.ascontiguousarray(ranks, dtype=np.int32)
    p = np.ascontiguousarray(ptl, dtype=np.float64)
    out = C.c_double()
    _check(load_library().darts_rollout_cost_dp(_np_ptr(ln), _np_ptr(rk), len(ln), n_ranks, _np_ptr(p),
                                                C.byref(out)))
    return out.value


def darts_fit_ptl(bsz, lat):
    import numpy as np
    b = np.ascontiguousarray(bsz, dtype=np.int32)
    y = np.ascontiguousarray(lat, dtype=np.float64)
    out = np.zeros(6, dtype=np.float64)
    _check(load_library().darts_fit_ptl(_np_ptr(b), _np_ptr(y), len(b), _np_ptr(out)))
    return tuple(float(x) for x in out)


# ---------------------------------------------------------------- stateful
def model_cfg_struct(model, weights=None):
    """weights: None, or a ctypes array of device pointers (weight_pointer_array)."""
    return ModelCfg(model.n_layers, model.d_model, model.n_q_heads, model.n_kv_heads,
                    model.head_dim, model.ffn_dim, model.vocab, model.n_experts, model.top_k,
                    model.expert_ffn, model.rope_theta, model.rms_eps,
                    DARTS_BF16 if model.dtype == "bf16" else DARTS_F32, model.weight_seed,
                    C.cast(weights, C.c_void_p) if weights is not None else None)


def weight_pointer_array(tensors):
    """ctypes array of the data pointers of caller weight tensors (device
    tensors in the order darts_model_cfg.weights documents)."""
    arr = (C.c_void_p * len(tensors))()
    for i, t in enumerate(tensors):
        arr[i] = t.data_ptr()
    return arr


def darts_weight_count(model):
    mc = model_cfg_struct(model)
    return int(load_library().darts_weight_count(C.byref(mc)))


def run_cfg_struct(run, stream, flags=0, page_perm_seed=0, kv_pool_bytes=None, traj_base=0):
    pool = int(run.kv_pool_gb * (1 << 30)) if kv_pool_bytes is None else int(kv_pool_bytes)
    return RunCfg(run.n_prompts, run.prompt_len, run.cap, run.L, run.m_up or 0, 16, pool,
                  run.sample_seed, run.temperature, flags, page_perm_seed, stream, traj_base)


class Rollout:
    """One rollout batch on the GPU through the C ABI (darts_init / darts_prefill /
    darts_decode_step / darts_select_and_prune).  Output buffers are torch
    tensors on the current device; PyTorch only allocates them."""

    def __init__(self, model, run, flags=0, page_perm_seed=0, kv_pool_bytes=None, stream=None, traj_base=0,
                 weights=None):
        """weights: None (generated from model.weight_seed) or the caller's
        device tensors in the order of darts_model_cfg.weights; the library
        copies them during darts_init."""
        import torch
        self.torch = torch
        self.lib = load_library()
        self.model, self.run = model, run
        self.m, self.k = run.m, run.k
        self.n_traj = run.n_prompts * run.m
        self.stream = stream or torch.cuda.current_stream()
        w_arr = weight_pointer_array(weights) if weights is not None else None
        self._mc = model_cfg_struct(model, w_arr)
        self._rc = run_cfg_struct(run, self.stream.cuda_stream, flags, page_perm_seed, kv_pool_bytes, traj_base)
        ctx = C.c_void_p()
        _check(self.lib.darts_init(C.byref(self._mc), run.m, run.k, C.byref(self._rc), C.byref(ctx)))
        self._mc.weights = None   # the library copied the tensors and keeps no reference
        self.ctx = ctx
        dev = torch.device("cuda", torch.cuda.current_device())
        n = self.n_traj
        self.o_traj = torch.zeros(n, dtype=torch.int32, device=dev)
        self.o_tok = torch.zeros(n, dtype=torch.int32, device=dev)
        self.o_samp = torch.zeros(n, dtype=torch.int32, device=dev)
        self.o_lp = torch.zeros(n, dtype=torch.float32, device=dev)
        self.o_ent = torch.zeros(n, dtype=torch.float32, device=dev)
        self.o_fin = torch.zeros(n, dtype=torch.uint8, device=dev)
        self.kept = torch.full((run.n_prompts, run.k), -1, dtype=torch.int32, device=dev)
        self.done_step = torch.full((run.n_prompts,), -1, dtype=torch.int32, device=dev)
        self._out = StepOut(self.o_traj.data_ptr(), self.o_tok.data_ptr(), self.o_samp.data_ptr(),
                            self.o_lp.data_ptr(), self.o_ent.data_ptr(), self.o_fin.data_ptr(), 0)
        self.n_live = n
        self.n_done = 0

    def close(self):
        if self.ctx:
            self.lib.darts_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _rows(self):
        n = self._out.n_rows
        return dict(traj=self.o_traj[:n], token=self.o_tok[:n], sampled=self.o_samp[:n],
                    logprob=self.o_lp[:n], entropy=self.o_ent[:n], finished=self.o_fin[:n])

    def darts_set_plan(self, plan):
        """Per-prompt candidate counts M'_i (k <= M'_i <= m) for the next prefill."""
        import numpy as np
        pl = np.ascontiguousarray(plan, dtype=np.int32)
        assert len(pl) == self.run.n_prompts
        _check(self.lib.darts_set_plan(self.ctx, _np_ptr(pl)), self.ctx)
        self.n_live = int(pl.sum())

    def darts_prefill(self, prompts, forced_len, force_tokens=None):
        _check(self.lib.darts_prefill(self.ctx, _ptr(prompts), _ptr(forced_len), _ptr(force_tokens),
                                      C.byref(self._out)), self.ctx)
        return self._rows()

    def darts_decode_step(self, force_tokens=None):
        _check(self.lib.darts_decode_step(self.ctx, _ptr(force_tokens), C.byref(self._out)), self.ctx)
        return self._rows()

    def darts_select_and_prune(self):
        nl, nd = C.c_int32(), C.c_int32()
        _check(self.lib.darts_select_and_prune(self.ctx, _ptr(self.kept), _ptr(self.done_step),
                                               C.byref(nl), C.byref(nd)), self.ctx)
        self.n_live, self.n_done = nl.value, nd.value
        return self.n_live, self.n_done

    def darts_reset(self):
        _check(self.lib.darts_reset(self.ctx), self.ctx)
        self.n_live, self.n_done = self.n_traj, 0
        self.kept.fill_(-1)
        self.done_step.fill_(-1)

    def stats(self):
        s = Stats()
        _check(self.lib.darts_get_stats(self.ctx, C.byref(s)), self.ctx)
        out = {}
        for f, _ in Stats._fields_:
            v = getattr(s, f)
            out[f] = list(v) if (f.startswith("gemm_cls") or f.startswith("moe_expert")) else v
        return out

    def step_times(self):
        """(rows per decode step, ms per decode step, prefill ms); needs FLAG_STEP_TIMES."""
        import numpy as np
        n = C.c_int32()
        pf = C.c_float()
        _check(self.lib.darts_get_step_times(self.ctx, None, None, 0, C.byref(n), C.byref(pf)), self.ctx)
        rows = np.zeros(n.value, np.int32)
        ms = np.zeros(n.value, np.float32)
        _check(self.lib.darts_get_step_times(self.ctx, _np_ptr(rows), _np_ptr(ms), n.value, C.byref(n),
                                             C.byref(pf)), self.ctx)
        return rows, ms, pf.value

    def stream_chunks(self, threshold, flush=False, out_cap=None):
        """Dispatch pending token chunks (FLAG_STREAM).  Returns None if nothing
        was dispatched, else (descriptors [n, 4] int32, tokens, log-probs) on
        the host; descriptor = (trajectory, start, count, final status)."""
        t = self.torch
        dev = self.o_tok.device
        cap = self.n_traj * self.run.cap if out_cap is None else out_cap
        if not hasattr(self, "_s_desc"):
            self._s_desc = t.zeros(self.n_traj * 4, dtype=t.int32, device=dev)
        if getattr(self, "_s_cap", -1) < cap:
            self._s_tok = t.zeros(max(cap, 1), dtype=t.int32, device=dev)
            self._s_lp = t.zeros(max(cap, 1), dtype=t.float32, device=dev)
            self._s_cap = cap
        nd, ntok = C.c_int32(), C.c_int64()
        _check(self.lib.darts_stream_chunks(self.ctx, threshold, int(flush), _ptr(self._s_desc),
                                            _ptr(self._s_tok), _ptr(self._s_lp), cap, C.byref(nd),
                                            C.byref(ntok)), self.ctx)
        if nd.value == 0:
            return None
        return (self._s_desc[:4 * nd.value].view(-1, 4).cpu().numpy(),
                self._s_tok[:ntok.value].cpu().numpy(), self._s_lp[:ntok.value].cpu().numpy())

    def traj_scores(self):
        t = self.torch
        dev = self.o_tok.device
        ln = t.zeros(self.n_traj, dtype=t.int32, device=dev)
        slp = t.zeros(self.n_traj, dtype=t.float32, device=dev)
        mlp = t.zeros(self.n_traj, dtype=t.float32, device=dev)
        st = t.zeros(self.n_traj, dtype=t.uint8, device=dev)
        _check(self.lib.darts_get_traj_scores(self.ctx, _ptr(ln), _ptr(slp), _ptr(mlp), _ptr(st)), self.ctx)
        return ln, slp, mlp, st

    def debug_moe_routing(self, force_ids=None, own_ids=None, used_p=None):
        """Routing verification buffers ([keys][n_layers][top_k] device tensors,
        int32 / int32 / float32; None turns a buffer off)."""
        ts = [t for t in (force_ids, own_ids, used_p) if t is not None]
        n_keys = ts[0].shape[0] if ts else 0
        _check(self.lib.darts_debug_moe_routing(self.ctx, _ptr(force_ids), _ptr(own_ids), _ptr(used_p),
                                                n_keys), self.ctx)

    def debug_fill_kv(self, byte):
        """Set every byte of the KV pools (before prefill; 0xff = NaN everywhere)."""
        _check(self.lib.darts_debug_fill_kv(self.ctx, int(byte)), self.ctx)

    def debug_logits(self, rows):
        t = self.torch
        buf = t.empty((rows, self.model.vocab), dtype=t.float32, device=self.o_tok.device)
        n = C.c_int32()
        _check(self.lib.darts_debug_logits(self.ctx, _ptr(buf), C.byref(n)), self.ctx)
        return buf[:n.value]

    def run_to_completion(self, prompts, forced_len, on_step=None, force_fn=None, plan=None):
        """prefill, then decode + select until every prompt's kept set is complete.
        on_step(step_index, rows) is called after every sampling step;
        force_fn(step_index) may return a [n_traj] int32 device tensor;
        plan: optional per-prompt candidate counts (darts_set_plan)."""
        if plan is not None:
            self.darts_set_plan(plan)
        rows = self.darts_prefill(prompts, forced_len, force_fn(0) if force_fn else None)
        if on_step:
            on_step(0, rows)
        self.darts_select_and_prune()
        s = 0
        while self.n_done < self.run.n_prompts:
            s += 1
            rows = self.darts_decode_step(force_fn(s) if force_fn else None)
            if on_step:
                on_step(s, rows)
            self.darts_select_and_prune()
        return self.stats()
