"""ctypes marshalling for include/rollout.h and include/sagc.h.  No computation
happens here."""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_PKG, "librollout.so")
_lib = None

RG_OK, RG_EINVAL, RG_ENOMEM, RG_EHIP, RG_EUNSUPPORTED = 0, -1, -2, -3, -4
RG_DTYPE_F32, RG_DTYPE_BF16 = 0, 1
RG_FLAG_NO_PREFIX_SHARING, RG_FLAG_PROFILE, RG_FLAG_GROUP_PREFIX, RG_FLAG_NO_ROW_TILES = 1, 2, 4, 8
KERNEL_KINDS = ["embed", "rmsnorm", "gemm_qkv", "qkv_rope", "attn", "attn_merge", "gemm_o", "gemm_gu", "swiglu",
                "gemm_down", "residual", "gemm_lm", "sample", "compact", "setup", "logprob"]

EXPORTS = ["rg_last_error", "rg_policy_create", "rg_policy_destroy", "rg_policy_device_bytes", "rollout_group",
           "group_advantage", "rg_philox_blocks", "rg_gumbel_bits", "rg_hbm_probe", "rg_step_history", "rg_kernel_times",
           "sagc_init", "sagc_group_stats", "sagc_step", "sagc_beta_draw", "group_filter",
           "recompute_logprobs", "grpo_surrogate", "rg_decode_attention_chunks", "rg_phase_times",
           "grpo_surrogate_noalloc"]
SAGC_MAX_SIZES = 8


def _pack_prompts(prompts):
    """A device int32 [P, Lp] tensor or a list of 1-D ones -> (packed, lengths)."""
    import torch
    if isinstance(prompts, torch.Tensor):
        _dev("prompts", prompts, torch.int32, ndim=2)
        if prompts.shape[0] < 1 or prompts.shape[1] < 1:
            raise ValueError("prompts must hold at least one prompt of at least one token")
        plen = [int(prompts.shape[1])] * int(prompts.shape[0])
        packed = prompts.view(-1)
    else:
        prompts = list(prompts)
        if not prompts:
            raise ValueError("prompts must hold at least one prompt")
        for i, p in enumerate(prompts):
            _dev(f"prompts[{i}]", p, torch.int32, ndim=1)
            if p.numel() < 1:
                raise ValueError(f"prompts[{i}] is empty")
        if len({p.device for p in prompts}) > 1:
            raise TypeError("prompts must all be in GPU memory")
        plen = [int(p.numel()) for p in prompts]
        packed = torch.cat(prompts)
    return packed, plen


class RolloutError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


class rg_config(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn_dim", C.c_int32), ("vocab", C.c_int32),
                ("eos_id", C.c_int32), ("rope_theta", C.c_float), ("rms_eps", C.c_float), ("dtype", C.c_int32)]


_PP = C.POINTER(C.c_void_p)


class rg_weights(C.Structure):
    _fields_ = [("embed", C.c_void_p), ("final_norm", C.c_void_p), ("lm_head", C.c_void_p),
                ("attn_norm", _PP), ("wq", _PP), ("wk", _PP), ("wv", _PP), ("wo", _PP), ("ffn_norm", _PP),
                ("w_gate", _PP), ("w_up", _PP), ("w_down", _PP)]


class rg_limits(C.Structure):
    _fields_ = [("max_seqs", C.c_int32), ("max_prompts", C.c_int32), ("max_prompt_tokens", C.c_int32),
                ("max_context", C.c_int32), ("kv_pool_pages", C.c_int64)]


class rg_sampling(C.Structure):
    _fields_ = [("temperature", C.c_float), ("flags", C.c_int32), ("forced_len", C.POINTER(C.c_int32)),
                ("force_tokens", C.c_void_p), ("dump_logits", C.c_void_p), ("dump_steps", C.c_int32),
                ("profile_kinds", C.c_uint32)]


class sagc_config(C.Structure):
    _fields_ = [("n_sizes", C.c_int32), ("sizes", C.c_int32 * SAGC_MAX_SIZES), ("tau", C.c_double),
                ("delta", C.c_double), ("eta", C.c_double), ("gamma", C.c_double), ("seed", C.c_uint64)]


class sagc_state(C.Structure):
    _fields_ = [("lam", C.c_double), ("alpha", C.c_double * SAGC_MAX_SIZES), ("beta", C.c_double * SAGC_MAX_SIZES),
                ("g_index", C.c_int32), ("reserved", C.c_int32), ("step", C.c_int64), ("last_rate", C.c_double),
                ("last_sample", C.c_double * SAGC_MAX_SIZES), ("last_score", C.c_double * SAGC_MAX_SIZES)]


def lib_path() -> str:
    return _LIB_PATH


def load_library():
    """Load librollout.so; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is missing: build it with `python -m paper_2606_02218_amd.build` "
                          "(or __graft_entry__.build()); there is no fallback path")
    lib = C.CDLL(_LIB_PATH)
    lib.rg_last_error.restype = C.c_char_p
    lib.rg_policy_create.argtypes = [C.POINTER(rg_config), C.POINTER(rg_weights), C.POINTER(rg_limits),
                                     C.POINTER(C.c_void_p)]
    lib.rg_policy_destroy.argtypes = [C.c_void_p]
    lib.rg_policy_destroy.restype = None
    lib.rg_policy_device_bytes.argtypes = [C.c_void_p]
    lib.rg_policy_device_bytes.restype = C.c_int64
    lib.rollout_group.argtypes = [C.c_void_p, C.c_void_p, C.POINTER(C.c_int32), C.c_int32, C.POINTER(C.c_int32),
                                  C.c_int32, C.c_uint64, C.POINTER(rg_sampling), C.c_void_p, C.c_void_p, C.c_void_p,
                                  C.c_void_p]
    lib.group_advantage.argtypes = [C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_float, C.c_int32, C.c_void_p,
                                    C.c_void_p]
    lib.rg_philox_blocks.argtypes = [C.c_uint64, C.c_uint64, C.c_void_p, C.c_int64, C.c_void_p, C.c_void_p]
    lib.rg_gumbel_bits.argtypes = [C.c_uint64, C.c_int32, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p]
    lib.rg_hbm_probe.argtypes = [C.c_void_p, C.c_void_p, C.c_int64, C.c_int32, C.c_int32, C.c_void_p]
    lib.rg_step_history.argtypes = [C.c_void_p, C.c_int32, C.POINTER(C.c_int32), C.c_void_p, C.c_void_p, C.c_void_p]
    lib.rg_kernel_times.argtypes = [C.c_void_p, C.c_int32, C.c_int32, C.POINTER(C.c_double), C.POINTER(C.c_int64)]
    lib.group_filter.argtypes = [C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p,
                                 C.c_void_p]
    lib.recompute_logprobs.argtypes = [C.c_void_p, C.c_void_p, C.POINTER(C.c_int32), C.c_int32, C.POINTER(C.c_int32),
                                       C.c_void_p, C.c_void_p, C.c_int32, C.c_float, C.c_int32, C.c_void_p, C.c_void_p]
    lib.grpo_surrogate.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32, C.c_int32,
                                   C.c_int32, C.c_void_p, C.c_double, C.c_double, C.c_int32, C.c_void_p, C.c_void_p]
    lib.rg_phase_times.argtypes = [C.c_void_p, C.POINTER(C.c_double), C.POINTER(C.c_double)]
    lib.rg_decode_attention_chunks.argtypes = [C.c_int32, C.c_int32, C.c_int32]
    lib.rg_decode_attention_chunks.restype = C.c_int32
    lib.grpo_surrogate_noalloc.argtypes = lib.grpo_surrogate.argtypes
    lib.sagc_init.argtypes = [C.POINTER(sagc_config), C.POINTER(sagc_state)]
    lib.sagc_group_stats.argtypes = [C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_double, C.c_void_p,
                                     C.c_void_p]
    lib.sagc_step.argtypes = [C.POINTER(sagc_config), C.POINTER(sagc_state), C.POINTER(C.c_float), C.c_int32,
                              C.POINTER(C.c_int32)]
    lib.sagc_beta_draw.argtypes = [C.c_uint64, C.c_int64, C.c_int32, C.c_double, C.c_double, C.POINTER(C.c_double)]
    _lib = lib
    return lib


def exported_symbols() -> list:
    lib = load_library()
    return [n for n in EXPORTS if hasattr(lib, n)]


def _check(rc: int):
    if rc != RG_OK:
        raise RolloutError(rc, load_library().rg_last_error().decode())


def _stream_ptr(stream=None) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _dev(name: str, t, dtype, shape=None, ndim=None):
    """Checks that ``t`` is a contiguous tensor of ``dtype`` (a torch dtype or
    a tuple of them) with ``shape`` (or ``ndim`` dimensions), in that order,
    so that no kernel reads or writes past a buffer the caller sized
    differently.  Raises TypeError / ValueError; returns ``t``.  Where it sits
    (GPU memory) is checked by _gpu once every argument has passed this."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor, got {type(t).__name__}")
    dts = dtype if isinstance(dtype, tuple) else (dtype,)
    if t.dtype not in dts:
        raise TypeError(f"{name} must have dtype {' or '.join(str(d) for d in dts)}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimension(s), got shape {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _gpu(**tensors):
    """Every named tensor (None skipped) must be in GPU memory."""
    for name, t in tensors.items():
        if t is not None and t.device.type != "cuda":
            raise TypeError(f"{name} must be in GPU memory, got device {t.device}")


class Policy:
    """A decoder loaded into librollout (the library copies the weights)."""

    def __init__(self, shape, weights, max_seqs: int, max_prompts: int, max_prompt_tokens: int, max_context: int,
                 kv_pool_pages: int = 0, device: str = "cuda"):
        import torch
        lib = load_library()
        self.shape = shape
        self.device = torch.device(device)
        dt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
        cfg = rg_config(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                        shape.ffn_dim, shape.vocab, shape.eos_id, float(shape.rope_theta), float(shape.rms_eps),
                        RG_DTYPE_BF16 if shape.dtype == "bf16" else RG_DTYPE_F32)
        keep = []

        def up(a, dtype):
            t = torch.from_numpy(np.ascontiguousarray(a)).to(device=self.device).to(dtype)
            keep.append(t)
            return t.data_ptr()

        def arr(name, dtype):
            a = (C.c_void_p * shape.n_layers)(*[up(lw[name], dtype) for lw in weights.layers])
            keep.append(a)
            return C.cast(a, _PP)

        w = rg_weights(up(weights.embed, dt), up(weights.final_norm, torch.float32), up(weights.lm_head, dt),
                       arr("attn_norm", torch.float32), arr("wq", dt), arr("wk", dt), arr("wv", dt), arr("wo", dt),
                       arr("ffn_norm", torch.float32), arr("w_gate", dt), arr("w_up", dt), arr("w_down", dt))
        lim = rg_limits(max_seqs, max_prompts, max_prompt_tokens, max_context, kv_pool_pages)
        h = C.c_void_p()
        torch.cuda.synchronize()
        _check(lib.rg_policy_create(C.byref(cfg), C.byref(w), C.byref(lim), C.byref(h)))
        torch.cuda.synchronize()
        del keep
        self._h = h
        self.limits = lim

    def close(self):
        if getattr(self, "_h", None):
            load_library().rg_policy_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def device_bytes(self) -> int:
        return int(load_library().rg_policy_device_bytes(self._h))

    def rollout(self, prompts, G: Sequence[int], max_new: int, seed: int, temperature: float = 1.0,
                forced_len=None, force_tokens=None, dump_steps: int = 0, share_prefix: bool = True,
                group_prefix_pass: bool = False, profile=False, out=None, stream=None):
        """prompts: device int32 tensor [P, Lp] or a list of 1-D device int32
        tensors.  Returns (tokens [N, max_new], lengths [N], logprobs
        [N, max_new]) and, with dump_steps, the logits [dump_steps, N, V].
        ``profile``: False, True (time every kernel class) or an iterable of
        class names from KERNEL_KINDS to time.  ``group_prefix_pass=True``
        makes bf16 models attend to each prompt's shared prefix once per group
        (RG_FLAG_GROUP_PREFIX)."""
        import torch
        lib = load_library()
        packed, plen = _pack_prompts(prompts)
        P = len(plen)
        G = [int(g) for g in G]
        if len(G) != P:
            raise ValueError(f"G must have one entry per prompt ({P}), got {len(G)}")
        N = sum(G)
        max_new = int(max_new)
        dev = packed.device
        if out is not None:
            tokens, lengths, logprobs = out
            _dev("tokens (out)", tokens, torch.int32, (N, max_new))
            _dev("lengths (out)", lengths, torch.int32, (N,))
            _dev("logprobs (out)", logprobs, torch.float32, (N, max_new))
        flags = ((0 if share_prefix else RG_FLAG_NO_PREFIX_SHARING) | (RG_FLAG_PROFILE if profile else 0)
                 | (RG_FLAG_GROUP_PREFIX if group_prefix_pass else 0))
        kinds = 0
        if profile and profile is not True:
            for name in profile:
                kinds |= 1 << KERNEL_KINDS.index(name)
        fl = None
        if forced_len is not None:
            if hasattr(forced_len, "detach"):
                forced_len = forced_len.detach().cpu().numpy()
            fl_np = np.ascontiguousarray(np.asarray(forced_len).reshape(-1))
            if fl_np.shape != (N,):
                raise ValueError(f"forced_len must have N = {N} entries, got {fl_np.size}")
            if not np.issubdtype(fl_np.dtype, np.integer):
                raise TypeError(f"forced_len must hold integers, got {fl_np.dtype}")
            fl_np = fl_np.astype(np.int32)
            fl = fl_np.ctypes.data_as(C.POINTER(C.c_int32))
        ft = None
        if force_tokens is not None:
            ft = _dev("force_tokens", force_tokens, torch.int32, (N, max_new))
        _gpu(prompts=packed, force_tokens=ft)
        if out is None:
            tokens = torch.empty((N, max_new), dtype=torch.int32, device=dev)
            lengths = torch.empty(N, dtype=torch.int32, device=dev)
            logprobs = torch.empty((N, max_new), dtype=torch.float32, device=dev)
        else:
            _gpu(tokens=tokens, lengths=lengths, logprobs=logprobs)
        dump = torch.empty((dump_steps, N, self.shape.vocab), dtype=torch.float32, device=dev) if dump_steps else None
        opts = rg_sampling(float(temperature), flags, fl, _ptr(ft), _ptr(dump), dump_steps, kinds)
        plen_a = (C.c_int32 * P)(*plen)
        g_a = (C.c_int32 * P)(*G)
        _check(lib.rollout_group(self._h, _ptr(packed), plen_a, P, g_a, max_new, C.c_uint64(seed & (2 ** 64 - 1)),
                                 C.byref(opts), _ptr(tokens), _ptr(lengths), _ptr(logprobs), _stream_ptr(stream)))
        if dump_steps:
            return tokens, lengths, logprobs, dump
        return tokens, lengths, logprobs

    def recompute_logprobs(self, prompts, G: Sequence[int], tokens, lengths, temperature: float = 1.0,
                           share_prefix: bool = True, row_tiles: bool = True, profile: bool = False, out=None,
                           stream=None):
        """Teacher-forced log-probabilities [N, max_new] of the completions
        ``tokens`` (device int32 [N, max_new]) with ``lengths`` (device int32
        [N]) after ``prompts`` (as for ``rollout``).  ``row_tiles=False``
        attends row by row (RG_FLAG_NO_ROW_TILES)."""
        import torch
        lib = load_library()
        packed, plen = _pack_prompts(prompts)
        P = len(plen)
        G = [int(g) for g in G]
        if len(G) != P:
            raise ValueError(f"G must have one entry per prompt ({P}), got {len(G)}")
        N = sum(G)
        _dev("tokens", tokens, torch.int32, ndim=2)
        if tokens.shape[0] != N:
            raise ValueError(f"tokens must have sum(G) = {N} rows, got {tokens.shape[0]}")
        max_new = int(tokens.shape[1])
        _dev("lengths", lengths, torch.int32, (N,))
        if out is not None:
            _dev("logprobs (out)", out, torch.float32, (N, max_new))
        _gpu(prompts=packed, tokens=tokens, lengths=lengths, out=out)
        lp = torch.empty((N, max_new), dtype=torch.float32, device=packed.device) if out is None else out
        flags = ((0 if share_prefix else RG_FLAG_NO_PREFIX_SHARING) | (RG_FLAG_PROFILE if profile else 0)
                 | (0 if row_tiles else RG_FLAG_NO_ROW_TILES))
        plen_a = (C.c_int32 * P)(*plen)
        g_a = (C.c_int32 * P)(*G)
        _check(lib.recompute_logprobs(self._h, _ptr(packed), plen_a, P, g_a, _ptr(tokens), _ptr(lengths), max_new,
                                      float(temperature), flags, _ptr(lp), _stream_ptr(stream)))
        return lp

    def step_history(self, cap: int = 1 << 16):
        lib = load_library()
        n = C.c_int32()
        a = np.zeros(cap, np.int32); g = np.zeros(cap, np.int32); c = np.zeros(cap, np.int64)
        _check(lib.rg_step_history(self._h, cap, C.byref(n), a.ctypes.data, g.ctypes.data, c.ctypes.data))
        k = min(cap, n.value)
        return a[:k].copy(), g[:k].copy(), c[:k].copy()

    def phase_times(self):
        """(prefill_ms, decode_ms) of the last rollout on the device timeline."""
        a, b = C.c_double(), C.c_double()
        _check(load_library().rg_phase_times(self._h, C.byref(a), C.byref(b)))
        return a.value, b.value

    def kernel_times(self, phase: int = 1) -> dict:
        lib = load_library()
        out = {}
        for i, name in enumerate(KERNEL_KINDS):
            ms = C.c_double(); n = C.c_int64()
            _check(lib.rg_kernel_times(self._h, phase, i, C.byref(ms), C.byref(n)))
            out[name] = (ms.value, n.value)
        return out


def group_advantage(rewards, G_dev, eps: float = 1e-6, ddof: int = 1, out=None, stream=None):
    """rewards: device fp32 [N]; G_dev: device int32 [P]."""
    import torch
    lib = load_library()
    _dev("rewards", rewards, torch.float32, ndim=1)
    _dev("G", G_dev, torch.int32, ndim=1)
    if out is not None:
        _dev("adv (out)", out, torch.float32, tuple(rewards.shape))
    _gpu(rewards=rewards, G=G_dev, out=out)
    if out is None:
        out = torch.empty_like(rewards)
    _check(lib.group_advantage(_ptr(rewards), _ptr(G_dev), int(G_dev.numel()), int(rewards.numel()), float(eps),
                               int(ddof), _ptr(out), _stream_ptr(stream)))
    return out


LOSS_MODES = {"token": 0, "seq": 1}


def grpo_surrogate(new_lp, old_lp, adv, lengths, G_dev, eps_lo: float = 0.2, eps_hi: float = 0.2,
                   mode: str = "token", keep=None, stream=None, out=None, noalloc: bool = False):
    """Clipped surrogate; returns a device fp64 tensor (loss, clipped
    fraction, counted tokens, counted sequences), written into ``out`` when
    given.  ``noalloc=True`` calls grpo_surrogate_noalloc (no device
    allocation in the library; N <= 65536)."""
    import torch
    lib = load_library()
    _dev("new_lp", new_lp, torch.float32, ndim=2)
    N, max_new = int(new_lp.shape[0]), int(new_lp.shape[1])
    _dev("old_lp", old_lp, torch.float32, (N, max_new))
    _dev("adv", adv, torch.float32, (N,))
    _dev("lengths", lengths, torch.int32, (N,))
    _dev("G", G_dev, torch.int32, ndim=1)
    if keep is not None:
        _dev("keep", keep, torch.int32, tuple(G_dev.shape))
    if mode not in LOSS_MODES:
        raise ValueError(f"mode must be one of {sorted(LOSS_MODES)}")
    if out is not None:
        _dev("out", out, torch.float64, (4,))
    _gpu(new_lp=new_lp, old_lp=old_lp, adv=adv, lengths=lengths, G=G_dev, keep=keep, out=out)
    if out is None:
        out = torch.empty(4, dtype=torch.float64, device=new_lp.device)
    fn = lib.grpo_surrogate_noalloc if noalloc else lib.grpo_surrogate
    _check(fn(_ptr(new_lp), _ptr(old_lp), _ptr(adv), _ptr(lengths), _ptr(G_dev), int(G_dev.numel()), N, max_new,
              _ptr(keep), float(eps_lo), float(eps_hi), LOSS_MODES[mode], _ptr(out), _stream_ptr(stream)))
    return out


def group_filter(rewards, G_dev, stream=None):
    """rewards: device fp32 [N]; G_dev: device int32 [P].  Returns device
    tensors (keep [P], kept_ids [P], n_kept [1]) as written by the library."""
    import torch
    lib = load_library()
    _dev("rewards", rewards, torch.float32, ndim=1)
    _dev("G", G_dev, torch.int32, ndim=1)
    _gpu(rewards=rewards, G=G_dev)
    P = int(G_dev.numel())
    keep = torch.empty(P, dtype=torch.int32, device=rewards.device)
    kept = torch.full((P,), -1, dtype=torch.int32, device=rewards.device)
    n = torch.empty(1, dtype=torch.int32, device=rewards.device)
    _check(lib.group_filter(_ptr(rewards), _ptr(G_dev), P, int(rewards.numel()), _ptr(keep), _ptr(kept), _ptr(n),
                            _stream_ptr(stream)))
    return keep, kept, n


def philox_blocks(key0: int, key1: int, ctr, stream=None):
    """ctr: device int64/uint64 tensor [n, 4] (bit patterns); returns [n, 4]."""
    import torch
    lib = load_library()
    _dev("ctr", ctr, (torch.int64, torch.uint64), ndim=2)
    if ctr.shape[1] != 4:
        raise ValueError(f"ctr must have shape [n, 4], got {tuple(ctr.shape)}")
    _gpu(ctr=ctr)
    out = torch.empty_like(ctr)
    _check(lib.rg_philox_blocks(C.c_uint64(key0), C.c_uint64(key1), _ptr(ctr), ctr.shape[0], _ptr(out),
                                _stream_ptr(stream)))
    return out


def hbm_probe(src, dst, mode: int, blocks: int = 2048, stream=None):
    """One launch of the streaming ceiling probe over the bytes of src (a
    contiguous device tensor, size a multiple of 16 bytes).  mode 1 copies to
    dst (same size); mode 0 reads only and dst must hold blocks * 256 int32."""
    lib = load_library()
    nbytes = src.numel() * src.element_size()
    if not src.is_contiguous() or not dst.is_contiguous():
        raise ValueError("src and dst must be contiguous")
    need = nbytes if mode == 1 else blocks * 256 * 4
    if dst.numel() * dst.element_size() < need:
        raise ValueError(f"dst must hold at least {need} bytes")
    _gpu(src=src, dst=dst)
    _check(lib.rg_hbm_probe(_ptr(src), _ptr(dst), C.c_int64(nbytes), mode, blocks, _stream_ptr(stream)))


def gumbel_bits(seed: int, t: int, s: int, vocab: int, stream=None):
    """Returns a device int32 tensor [vocab] holding the uint32 bit patterns."""
    import torch
    lib = load_library()
    out = torch.empty(vocab, dtype=torch.int32, device="cuda")
    _check(lib.rg_gumbel_bits(C.c_uint64(seed), t, s, vocab, _ptr(out), _stream_ptr(stream)))
    return out


class Sagc:
    """Straggler-aware group-size controller (include/sagc.h): host state,
    one step per rollout."""

    def __init__(self, sizes=(4, 8, 16), tau: float = 1.25, delta: float = 0.1, eta: float = 0.5,
                 gamma: float = 0.95, seed: int = 0):
        lib = load_library()
        sizes = [int(s) for s in sizes]
        if not 1 <= len(sizes) <= SAGC_MAX_SIZES:
            raise ValueError("between 1 and 8 sizes")
        arr = (C.c_int32 * SAGC_MAX_SIZES)(*(sizes + [0] * (SAGC_MAX_SIZES - len(sizes))))
        self.cfg = sagc_config(len(sizes), arr, float(tau), float(delta), float(eta), float(gamma),
                               C.c_uint64(seed & (2 ** 64 - 1)))
        self.sizes = sizes
        self.state = sagc_state()
        _check(lib.sagc_init(C.byref(self.cfg), C.byref(self.state)))

    @property
    def G(self) -> int:
        return self.sizes[self.state.g_index]

    def group_stats(self, lengths, G_dev, out=None, stream=None):
        """lengths: device int32 [N]; G_dev: device int32 [P].  Returns device
        float [P, 4] = (l_max, l_median, R, S)."""
        import torch
        lib = load_library()
        _dev("lengths", lengths, torch.int32, ndim=1)
        _dev("G", G_dev, torch.int32, ndim=1)
        P = int(G_dev.numel())
        if out is None:
            out = torch.empty((P, 4), dtype=torch.float32, device=lengths.device)
        else:
            _dev("stats (out)", out, torch.float32, (P, 4))
        _gpu(lengths=lengths, G=G_dev, out=out)
        _check(lib.sagc_group_stats(_ptr(lengths), _ptr(G_dev), P, int(lengths.numel()), self.cfg.tau, _ptr(out),
                                    _stream_ptr(stream)))
        return out

    def step(self, stats) -> int:
        """stats: [n_groups, 4] (host numpy or any tensor; column 3 = S).
        Returns the next group size."""
        lib = load_library()
        if hasattr(stats, "detach"):
            stats = stats.detach().cpu().numpy()
        s = np.ascontiguousarray(np.asarray(stats, dtype=np.float32).reshape(-1, 4))
        g = C.c_int32()
        _check(lib.sagc_step(C.byref(self.cfg), C.byref(self.state), s.ctypes.data_as(C.POINTER(C.c_float)),
                             s.shape[0], C.byref(g)))
        return g.value

    def snapshot(self) -> dict:
        k = len(self.sizes)
        st = self.state
        return {"lambda": st.lam, "alpha": list(st.alpha[:k]), "beta": list(st.beta[:k]), "g_index": st.g_index,
                "step": st.step, "last_rate": st.last_rate, "last_sample": list(st.last_sample[:k]),
                "last_score": list(st.last_score[:k])}


def decode_attention_chunks(rows: int, n_kv: int, ctx_max: int) -> int:
    """Context chunks per row of a decode step's attention (see rollout.h)."""
    n = load_library().rg_decode_attention_chunks(int(rows), int(n_kv), int(ctx_max))
    _check(min(n, 0))
    return n


def sagc_beta_draw(seed: int, step: int, arm: int, a: float, b: float) -> float:
    lib = load_library()
    out = C.c_double()
    _check(lib.sagc_beta_draw(C.c_uint64(seed & (2 ** 64 - 1)), step, arm, a, b, C.byref(out)))
    return out.value
