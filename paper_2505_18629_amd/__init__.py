"""Python binding of librv.so, the gfx950 Reflective Verification verify pass.

Every function mirrors the C ABI of include/rv.h under the same name and only
marshals arguments: device buffers are torch CUDA tensors (their data_ptr is
passed), host arrays are Python sequences or numpy arrays, and the stream is
torch's current stream unless one is given.  All compute runs in the HIP
kernels of the library; there is no fallback.  Importing this module raises
if the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librv.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with paper_2505_18629_amd.build.build()")

# torch first: its HIP runtime (soname libamdhip64.so.7) is then the one the
# library binds to, so there is a single runtime and device context per process.
import torch  # noqa: E402,F401

_lib = ctypes.CDLL(LIB_PATH)

RV_F32, RV_BF16 = 0, 1
RV_RULE_GREEDY, RV_RULE_TYPICAL, RV_RULE_SAMPLING = 0, 1, 2
RV_ENTROPY_FUSED, RV_ENTROPY_ORIGINAL = 0, 1
RV_MAX_BATCH, RV_MAX_DRAFTS = 256, 32
(RV_OUT_ORIG, RV_OUT_REFL, RV_OUT_FUSED, RV_OUT_LOGP_ORIG, RV_OUT_LOGP_REFL, RV_OUT_LOGP_FUSED, RV_OUT_ENTROPY,
 RV_OUT_MARGINS, RV_OUT_PROB_FUSED) = range(9)
RV_MAT_QKV, RV_MAT_O, RV_MAT_GATEUP, RV_MAT_DOWN, RV_MAT_LM_HEAD = range(5)
RV_WS_RESID, RV_WS_ATTN, RV_WS_ACT, RV_WS_QUERY = range(4)
PROF_CLASSES = ["plan", "norm", "qkv", "attn", "combine", "o", "gateup", "down", "lmhead", "tail"]
STATUS = {0: "RV_OK", -1: "RV_E_ARG", -2: "RV_E_RANGE", -3: "RV_E_CAPACITY", -4: "RV_E_BUFFER",
          -5: "RV_E_HIP", -6: "RV_E_STATE"}

EXPORTED = [
    "rv_status_str", "rv_last_error", "rv_model_bytes", "rv_init_weights", "rv_model_free",
    "rv_cache_bytes", "rv_cache_create", "rv_cache_free", "rv_prefill_cache", "rv_verify", "rv_verify_sampled",
    "rv_verify_ragged", "rv_commit_tokens", "rv_fuse_accept_noalloc",
    "rv_debug_fuse_accept", "rv_debug_output", "rv_debug_export_kv", "rv_debug_export_ids", "rv_debug_weight_bits",
    "rv_debug_linear", "rv_debug_workspace", "rv_debug_profile", "rv_debug_profile_read", "rv_debug_time_matrix",
]


class rv_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("dtype", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_base", ctypes.c_float), ("init_std", ctypes.c_float)]


class rv_fusion(ctypes.Structure):
    _fields_ = [("alpha", ctypes.c_float), ("prefix_pos", ctypes.c_int32), ("rule", ctypes.c_int32),
                ("epsilon", ctypes.c_float), ("delta", ctypes.c_float), ("entropy_src", ctypes.c_int32),
                ("temperature", ctypes.c_float)]


class RVError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status
        self.name = STATUS.get(status, str(status))


_vp, _i32, _u64, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64, ctypes.c_size_t
_P_i32 = ctypes.POINTER(ctypes.c_int32)
_sig = {
    "rv_status_str": ([ctypes.c_int], ctypes.c_char_p),
    "rv_last_error": ([], ctypes.c_char_p),
    "rv_model_bytes": ([ctypes.POINTER(rv_config), ctypes.POINTER(_sz)], ctypes.c_int),
    "rv_init_weights": ([ctypes.POINTER(rv_config), _u64, _vp, _sz, _vp, ctypes.POINTER(_vp)], ctypes.c_int),
    "rv_model_free": ([_vp], None),
    "rv_cache_bytes": ([_vp, _i32, _i32, _i32, _i32, ctypes.POINTER(_sz)], ctypes.c_int),
    "rv_cache_create": ([_vp, _i32, _i32, _i32, _i32, _vp, _sz, ctypes.POINTER(_vp)], ctypes.c_int),
    "rv_cache_free": ([_vp], None),
    "rv_prefill_cache": ([_vp, _vp, _i32, _P_i32, _vp], ctypes.c_int),
    "rv_verify": ([_vp, _P_i32, _vp, _i32, _vp, _i32, ctypes.POINTER(rv_fusion), _vp, _vp, _vp], ctypes.c_int),
    "rv_verify_sampled": ([_vp, _P_i32, _vp, _i32, _vp, _vp, _i32, ctypes.POINTER(rv_fusion), ctypes.c_uint64, _vp,
                           _vp, _vp], ctypes.c_int),
    "rv_commit_tokens": ([_vp, _P_i32, _vp, _vp], ctypes.c_int),
    "rv_verify_ragged": ([_vp, _P_i32, _vp, _i32, _P_i32, _vp, _i32, ctypes.POINTER(rv_fusion), _vp, _vp, _vp],
                         ctypes.c_int),
    "rv_fuse_accept_noalloc": ([_vp, _i32, _i32, _i32, _vp, ctypes.POINTER(rv_fusion), _vp, _vp, _vp], ctypes.c_int),
    "rv_debug_fuse_accept": ([_vp, _vp, _P_i32, _vp, _i32, ctypes.POINTER(rv_fusion), _vp, _vp, _vp], ctypes.c_int),
    "rv_debug_output": ([_vp, _i32, _vp, _sz, _vp], ctypes.c_int),
    "rv_debug_export_kv": ([_vp, _i32, _i32, _i32, _i32, _vp, _vp, _sz, _vp], ctypes.c_int),
    "rv_debug_export_ids": ([_vp, _i32, _i32, _i32, _vp, _vp], ctypes.c_int),
    "rv_debug_weight_bits": ([_vp, _i32, _vp, _i32, _vp], ctypes.c_int),
    "rv_debug_linear": ([_vp, _i32, _i32, _vp, _i32, _vp, _sz, _vp], ctypes.c_int),
    "rv_debug_workspace": ([_vp, _i32, _i32, _vp, _sz, _vp], ctypes.c_int),
    "rv_debug_profile": ([_vp, _i32], ctypes.c_int),
    "rv_debug_time_matrix": ([_vp, _i32, _i32, _i32, _vp, ctypes.POINTER(ctypes.c_float)], ctypes.c_int),
    "rv_debug_profile_read": ([_vp, _i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_i32)], ctypes.c_int),
}
for _name, (_args, _res) in _sig.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = _res


def _check(status: int) -> None:
    if status != 0:
        raise RVError(status, _lib.rv_last_error().decode())


def _dev(t) -> Optional[int]:
    """Device pointer of a torch tensor (or None)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    import torch
    return torch.cuda.current_stream().cuda_stream


def _host_i32(vals: Sequence[int]):
    arr = np.ascontiguousarray(np.asarray(vals, dtype=np.int32))
    return arr, arr.ctypes.data_as(_P_i32)


def make_config(shape) -> rv_config:
    """rv_config of a model shape (any object with the ModelShape fields)."""
    return rv_config(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim,
                     shape.ffn_dim, shape.vocab, RV_BF16 if shape.dtype == "bf16" else RV_F32,
                     shape.rms_eps, shape.rope_base, shape.init_std)


# ------------------------------------------------------------------- C ABI

def rv_status_str(status: int) -> str:
    return _lib.rv_status_str(status).decode()


def rv_last_error() -> str:
    return _lib.rv_last_error().decode()


def rv_model_bytes(cfg: rv_config) -> int:
    n = _sz()
    _check(_lib.rv_model_bytes(ctypes.byref(cfg), ctypes.byref(n)))
    return n.value


def rv_init_weights(cfg: rv_config, seed: int, buf, stream=None) -> int:
    h = _vp()
    _check(_lib.rv_init_weights(ctypes.byref(cfg), seed, _dev(buf), buf.numel() * buf.element_size(),
                                _stream(stream), ctypes.byref(h)))
    return h.value


def rv_model_free(model: int) -> None:
    _lib.rv_model_free(model)


def rv_cache_bytes(model: int, batch: int, max_len: int, max_block: int, max_drafts: int) -> int:
    n = _sz()
    _check(_lib.rv_cache_bytes(model, batch, max_len, max_block, max_drafts, ctypes.byref(n)))
    return n.value


def rv_cache_create(model: int, batch: int, max_len: int, max_block: int, max_drafts: int, buf) -> int:
    h = _vp()
    _check(_lib.rv_cache_create(model, batch, max_len, max_block, max_drafts, _dev(buf),
                                buf.numel() * buf.element_size(), ctypes.byref(h)))
    return h.value


def rv_cache_free(cache: int) -> None:
    _lib.rv_cache_free(cache)


def rv_prefill_cache(cache: int, prefix_ids, prefix_len: Sequence[int], stream=None) -> None:
    """prefix_ids: device int32 [batch][ld]; prefix_len: host lengths."""
    _keep, lens = _host_i32(prefix_len)
    _check(_lib.rv_prefill_cache(cache, _dev(prefix_ids), prefix_ids.shape[-1], lens, _stream(stream)))


def rv_verify(cache: int, prefix_len: Sequence[int], draft_ids, k: int, probe_ids, n_probe: int, alpha: float,
              prefix_pos: int, accept_len, next_id, rule: int = RV_RULE_GREEDY, stream=None,
              epsilon: float = 0.09, delta: float = 0.3, entropy_src: int = RV_ENTROPY_FUSED,
              temperature: float = 1.0) -> None:
    _keep, lens = _host_i32(prefix_len)
    fu = rv_fusion(alpha, prefix_pos, rule, epsilon, delta, entropy_src, temperature)
    _check(_lib.rv_verify(cache, lens, _dev(draft_ids), k, _dev(probe_ids), n_probe, ctypes.byref(fu),
                          _dev(accept_len), _dev(next_id), _stream(stream)))


def rv_verify_sampled(cache: int, prefix_len: Sequence[int], draft_ids, k: int, draft_probs, probe_ids,
                      n_probe: int, alpha: float, prefix_pos: int, seed: int, accept_len, next_id,
                      temperature: float = 1.0, rule: int = RV_RULE_SAMPLING, stream=None) -> None:
    _keep, lens = _host_i32(prefix_len)
    fu = rv_fusion(alpha, prefix_pos, rule, 0.0, 0.0, RV_ENTROPY_FUSED, temperature)
    _check(_lib.rv_verify_sampled(cache, lens, _dev(draft_ids), k, _dev(draft_probs), _dev(probe_ids), n_probe,
                                  ctypes.byref(fu), seed, _dev(accept_len), _dev(next_id), _stream(stream)))


def rv_verify_ragged(cache: int, prefix_len: Sequence[int], draft_ids, ld_drafts: int, draft_len: Sequence[int],
                     probe_ids, n_probe: int, alpha: float, prefix_pos: int, accept_len, next_id,
                     rule: int = RV_RULE_GREEDY, epsilon: float = 0.09, delta: float = 0.3,
                     entropy_src: int = RV_ENTROPY_FUSED, temperature: float = 1.0, stream=None) -> None:
    _keep, lens = _host_i32(prefix_len)
    _keep2, kl = _host_i32(draft_len)
    fu = rv_fusion(alpha, prefix_pos, rule, epsilon, delta, entropy_src, temperature)
    _check(_lib.rv_verify_ragged(cache, lens, _dev(draft_ids), ld_drafts, kl, _dev(probe_ids), n_probe,
                                 ctypes.byref(fu), _dev(accept_len), _dev(next_id), _stream(stream)))


def rv_commit_tokens(cache: int, positions: Sequence[int], ids, stream=None) -> None:
    _keep, pos = _host_i32(positions)
    _check(_lib.rv_commit_tokens(cache, pos, _dev(ids), _stream(stream)))


RV_NOALLOC_SCRATCH_BYTES = 4718592


def rv_fuse_accept_noalloc(logits, k: int, draft_ids, alpha: float, accept_len, next_id,
                           rule: int = RV_RULE_GREEDY, epsilon: float = 0.09, delta: float = 0.3,
                           entropy_src: int = RV_ENTROPY_FUSED, temperature: float = 1.0, stream=None) -> None:
    """logits: device fp32 [batch][2(k+1)][vocab]; no cache, scratch in the
    library's static device array."""
    fu = rv_fusion(alpha, 0, rule, epsilon, delta, entropy_src, temperature)
    _check(_lib.rv_fuse_accept_noalloc(_dev(logits), logits.shape[0], k, logits.shape[-1], _dev(draft_ids),
                                       ctypes.byref(fu), _dev(accept_len), _dev(next_id), _stream(stream)))


def rv_debug_fuse_accept(cache: int, logits, prefix_len: Sequence[int], draft_ids, k: int, alpha: float,
                         accept_len, next_id, rule: int = RV_RULE_GREEDY, epsilon: float = 0.09, delta: float = 0.3,
                         entropy_src: int = RV_ENTROPY_FUSED, temperature: float = 1.0, stream=None) -> None:
    """logits: device fp32 [batch][2(k+1)][vocab] (o rows, then r rows)."""
    _keep, lens = _host_i32(prefix_len)
    fu = rv_fusion(alpha, 0, rule, epsilon, delta, entropy_src, temperature)
    _check(_lib.rv_debug_fuse_accept(cache, _dev(logits), lens, _dev(draft_ids), k, ctypes.byref(fu),
                                     _dev(accept_len), _dev(next_id), _stream(stream)))


def rv_debug_output(cache: int, which: int, dst, stream=None) -> None:
    _check(_lib.rv_debug_output(cache, which, _dev(dst), dst.numel() * dst.element_size(), _stream(stream)))


def rv_debug_export_kv(cache: int, layer: int, seq: int, pos0: int, npos: int, dst_k, dst_v, stream=None) -> None:
    _check(_lib.rv_debug_export_kv(cache, layer, seq, pos0, npos, _dev(dst_k), _dev(dst_v),
                                   min(dst_k.numel() * dst_k.element_size(), dst_v.numel() * dst_v.element_size()),
                                   _stream(stream)))


def rv_debug_export_ids(cache: int, seq: int, pos0: int, n: int, dst, stream=None) -> None:
    _check(_lib.rv_debug_export_ids(cache, seq, pos0, n, _dev(dst), _stream(stream)))


def rv_debug_weight_bits(model: int, tensor: int, flat_idx) -> np.ndarray:
    idx = np.ascontiguousarray(np.asarray(flat_idx, dtype=np.int64))
    out = np.zeros(len(idx), dtype=np.uint32)
    _check(_lib.rv_debug_weight_bits(model, tensor, idx.ctypes.data, len(idx), out.ctypes.data))
    return out


def rv_debug_linear(cache: int, layer: int, matrix: int, x, y, stream=None) -> None:
    """x: operand rows [M][K] (fp32 models) or planes [2][M][K] (bf16 models)."""
    _check(_lib.rv_debug_linear(cache, layer, matrix, _dev(x), x.shape[-2], _dev(y),
                                y.numel() * y.element_size(), _stream(stream)))


def rv_debug_workspace(cache: int, which: int, rows: int, dst, stream=None) -> None:
    _check(_lib.rv_debug_workspace(cache, which, rows, _dev(dst), dst.numel() * dst.element_size(),
                                   _stream(stream)))


def rv_debug_profile(cache: int, enable: bool) -> None:
    _check(_lib.rv_debug_profile(cache, 1 if enable else 0))


def rv_debug_profile_read(cache: int, kclass: int):
    """(total ms, launches) of one kernel class since profiling was enabled."""
    ms, n = ctypes.c_double(), _i32()
    _check(_lib.rv_debug_profile_read(cache, kclass, ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def rv_debug_time_matrix(cache: int, matrix: int, M: int, reps: int, stream=None) -> float:
    """Average ms of the production kernel of one matrix class (synchronous)."""
    ms = ctypes.c_float()
    _check(_lib.rv_debug_time_matrix(cache, matrix, M, reps, _stream(stream), ctypes.byref(ms)))
    return ms.value


# ------------------------------------------------------------------- buffers

class Verifier:
    """Owns the device buffers (torch tensors) of one model and one cache and
    calls the C ABI on them.  Plumbing only."""

    def __init__(self, shape, seed: int, batch: int, max_len: int, max_block: int = 64,
                 max_drafts: int = 16, device: str = "cuda"):
        import torch
        self.torch = torch
        self.shape = shape
        self.cfg = make_config(shape)
        self.batch = batch
        self.model_buf = torch.empty(rv_model_bytes(self.cfg), dtype=torch.uint8, device=device)
        self.model = rv_init_weights(self.cfg, seed, self.model_buf)
        nbytes = rv_cache_bytes(self.model, batch, max_len, max_block, max_drafts)
        self.cache_buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
        torch.cuda.synchronize()
        self.cache = rv_cache_create(self.model, batch, max_len, max_block, max_drafts, self.cache_buf)
        self.accept_len = torch.zeros(batch, dtype=torch.int32, device=device)
        self.next_id = torch.zeros(batch, dtype=torch.int32, device=device)
        self.k = None

    def prefill(self, prefixes: Sequence[Sequence[int]]):
        torch = self.torch
        lens = [len(p) for p in prefixes]
        ld = max(lens)
        ids = np.zeros((self.batch, ld), dtype=np.int32)
        for b, p in enumerate(prefixes):
            ids[b, :len(p)] = p
        d_ids = torch.from_numpy(ids).cuda()
        rv_prefill_cache(self.cache, d_ids, lens)
        self._keep = d_ids
        return lens

    def verify_ragged(self, prefix_len, drafts: Sequence[Sequence[int]], probe, alpha: float, prefix_pos: int,
                      **kw):
        """One draft list per sequence (lengths may differ)."""
        torch = self.torch
        kl = [len(d) for d in drafts]
        ld = max(max(kl), 1)
        pad = np.zeros((self.batch, ld), dtype=np.int32)
        for b, d in enumerate(drafts):
            pad[b, :len(d)] = d
        d_dr = torch.from_numpy(pad).cuda()
        probe = np.asarray(probe, dtype=np.int32)
        d_pr = torch.from_numpy(probe).cuda() if len(probe) else None
        rv_verify_ragged(self.cache, prefix_len, d_dr, ld, kl, d_pr, len(probe), alpha, prefix_pos,
                         self.accept_len, self.next_id, **kw)
        self._keep2 = (d_dr, d_pr)
        self.k, self.kb = ld, kl
        return self.accept_len, self.next_id

    def verify_sampled(self, prefix_len, drafts, q, probe, alpha: float, prefix_pos: int, seed: int,
                       temperature: float = 1.0):
        """Algorithm 1's rule; q [batch][k][vocab] are the draft distributions."""
        torch = self.torch
        drafts = np.asarray(drafts, dtype=np.int32).reshape(self.batch, -1)
        k = drafts.shape[1]
        d_dr = torch.from_numpy(np.ascontiguousarray(drafts)).cuda()
        d_q = torch.from_numpy(np.ascontiguousarray(np.asarray(q, dtype=np.float32))).cuda() if k else None
        probe = np.asarray(probe, dtype=np.int32)
        d_pr = torch.from_numpy(probe).cuda() if len(probe) else None
        rv_verify_sampled(self.cache, prefix_len, d_dr, k, d_q, d_pr, len(probe), alpha, prefix_pos, seed,
                          self.accept_len, self.next_id, temperature=temperature)
        self._keep2 = (d_dr, d_pr, d_q)
        self.k, self.kb = k, None
        return self.accept_len, self.next_id

    def verify(self, prefix_len, drafts, probe, alpha: float, prefix_pos: int, rule: int = RV_RULE_GREEDY,
               epsilon: float = 0.09, delta: float = 0.3, entropy_src: int = RV_ENTROPY_FUSED,
               temperature: float = 1.0):
        torch = self.torch
        drafts = np.asarray(drafts, dtype=np.int32).reshape(self.batch, -1)
        k = drafts.shape[1]
        d_dr = torch.from_numpy(np.ascontiguousarray(drafts)).cuda()
        probe = np.asarray(probe, dtype=np.int32)
        d_pr = torch.from_numpy(probe).cuda() if len(probe) else None
        rv_verify(self.cache, prefix_len, d_dr, k, d_pr, len(probe), alpha, prefix_pos,
                  self.accept_len, self.next_id, rule=rule, epsilon=epsilon, delta=delta, entropy_src=entropy_src,
                  temperature=temperature)
        self._keep2 = (d_dr, d_pr)
        self.k, self.kb = k, None
        return self.accept_len, self.next_id

    def output(self, which: int):
        """Uniform draft counts: [batch][k+1] rows; ragged (verify_ragged):
        [sum(k_b+1)] rows, sequence after sequence."""
        torch = self.torch
        rows = (self.batch, self.k + 1) if getattr(self, "kb", None) is None else (sum(k + 1 for k in self.kb),)
        if which == RV_OUT_ENTROPY:
            shape = (2,) + rows
        elif which == RV_OUT_MARGINS:
            shape = (self.batch, self.k + 2)
        else:
            shape = rows + (self.shape.vocab,)
        out = torch.empty(shape, dtype=torch.float32, device="cuda")
        rv_debug_output(self.cache, which, out)
        return out

    def close(self):
        if getattr(self, "cache", None):
            rv_cache_free(self.cache)
            self.cache = None
        if getattr(self, "model", None):
            rv_model_free(self.model)
            self.model = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
