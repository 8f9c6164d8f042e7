"""MLKV decode attention on AMD Instinct MI355X (gfx950).

Thin ctypes binding of ``libmlkv.so`` (C ABI declared in ``include/mlkv.h``).
It only marshals arguments: torch tensors supply device memory and the HIP
stream, every step of the computation runs in the library's HIP kernels.
There is no fallback: if the library is missing, importing the binding
functions raises.

Paper: MLKV, Multi-Layer Key-Value heads (arXiv 2406.09297): GQA grouping
inside a layer (Section 2.3, Eq. 12) and KV-head sharing across consecutive
layers (Section 3, Eqs. 13-17); decode with a KV cache (Section 2.4).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch  # loaded first: the library then binds to torch's HIP runtime

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmlkv.so")

MLKV_OK = 0
STATUS_NAMES = ["MLKV_OK", "MLKV_ERR_INVALID_ARG", "MLKV_ERR_BAD_MAP", "MLKV_ERR_ALIGNMENT",
                "MLKV_ERR_UNSUPPORTED", "MLKV_ERR_CAPACITY", "MLKV_ERR_WORKSPACE", "MLKV_ERR_HIP"]
OUT_F32 = 0
OUT_BF16 = 1
V_BLOCK = 32  # tokens per channel-major block of the value plane

# Every symbol include/mlkv.h declares.
EXPORTS = [
    "mlkv_status_string", "mlkv_last_error", "mlkv_map_create_uniform", "mlkv_map_create",
    "mlkv_map_destroy", "mlkv_map_num_layers", "mlkv_map_num_q_heads", "mlkv_map_num_kv_heads",
    "mlkv_map_kv_head", "mlkv_map_owner_layer", "mlkv_map_layer_kv_count",
    "mlkv_map_layer_owned_count", "mlkv_map_layer_owned_begin", "mlkv_cache_bytes",
    "mlkv_workspace_bytes", "mlkv_cache_append", "mlkv_decode_attention", "mlkv_decode_step",
    "mlkv_plan", "mlkv_plan_merge_kernel", "mlkv_workspace_init", "mlkv_profile_enable", "mlkv_profile_read",
    "mlkv_profile_durations", "mlkv_profile_disable", "mlkv_profile_launch_floor",
    "mlkv_profile_read_bandwidth",
    "mlkv_decode_step_rope", "mlkv_workspace_bytes_rope", "mlkv_decode_step_noalloc",
    "mlkv_cache_append_rows", "mlkv_prefill_attention", "mlkv_prefill_step",
    "mlkv_cache_write_rows", "mlkv_cache_read_rows",
    "mlkv_model_create", "mlkv_model_destroy", "mlkv_model_workspace_bytes",
    "mlkv_model_fused_path",
    "mlkv_model_decode_step",
]


class MLKVError(RuntimeError):
    def __init__(self, status: int, message: str):
        name = STATUS_NAMES[status] if 0 <= status < len(STATUS_NAMES) else str(status)
        super().__init__(f"{name}: {message}")
        self.status = status
        self.status_name = name


class _Cache(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("n_kv", ctypes.c_int),
                ("batch", ctypes.c_int), ("capacity", ctypes.c_int), ("head_dim", ctypes.c_int)]


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                              "(hipcc, gfx950); there is no fallback implementation")
        L = ctypes.CDLL(LIB_PATH)
        P, I, Z, S = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t, ctypes.c_int
        sig = {
            "mlkv_status_string": ([I], ctypes.c_char_p),
            "mlkv_last_error": ([], ctypes.c_char_p),
            "mlkv_map_create_uniform": ([I, I, I, I, ctypes.POINTER(P)], S),
            "mlkv_map_create": ([I, I, I, P, P, ctypes.POINTER(P)], S),
            "mlkv_map_destroy": ([P], None),
            "mlkv_map_num_layers": ([P], I),
            "mlkv_map_num_q_heads": ([P], I),
            "mlkv_map_num_kv_heads": ([P], I),
            "mlkv_map_kv_head": ([P, I, I], I),
            "mlkv_map_owner_layer": ([P, I], I),
            "mlkv_map_layer_kv_count": ([P, I], I),
            "mlkv_map_layer_owned_count": ([P, I], I),
            "mlkv_map_layer_owned_begin": ([P, I], I),
            "mlkv_cache_bytes": ([P, I, I, I], Z),
            "mlkv_workspace_bytes": ([P, I, I, I], Z),
            "mlkv_cache_append": ([I, P, P, P, P, I, P, P], S),
            "mlkv_decode_attention": ([I, P, P, P, P, P, I, I, P, Z, P], S),
            "mlkv_decode_step": ([P, P, P, P, P, P, P, I, I, P, Z, P], S),
            "mlkv_decode_step_rope": ([P, P, P, P, P, P, I, ctypes.c_double, P, I, I, P, Z, P], S),
            "mlkv_workspace_bytes_rope": ([P, I, I, I, I], Z),
            "mlkv_decode_step_noalloc": ([P, P, P, P, P, P, P, I, I, P], S),
            "mlkv_cache_append_rows": ([I, P, P, P, P, I, I, P, P], S),
            "mlkv_cache_write_rows": ([P, I, I, P, P, P], S),
            "mlkv_cache_read_rows": ([P, I, I, P, P, P], S),
            "mlkv_prefill_attention": ([I, P, P, P, P, I, P, I, P], S),
            "mlkv_prefill_step": ([P, P, P, P, P, P, I, P, I, P], S),
            "mlkv_model_create": ([P, I, I, I, I, ctypes.c_double, ctypes.c_double, P, P], S),
            "mlkv_model_destroy": ([P], None),
            "mlkv_model_workspace_bytes": ([P, I, I], Z),
            "mlkv_model_fused_path": ([P, I], I),
            "mlkv_model_decode_step": ([P, P, P, P, I, P, Z, P], S),
            "mlkv_plan": ([P, I, I, I, I, I, ctypes.POINTER(I), ctypes.POINTER(I)], S),
            "mlkv_plan_merge_kernel": ([P, I, I, I, I, I], I),
            "mlkv_workspace_init": ([P, Z, P], S),
            "mlkv_profile_enable": ([I], S),
            "mlkv_profile_read": ([ctypes.POINTER(I)] + [ctypes.POINTER(ctypes.c_double)] * 3, S),
            "mlkv_profile_durations": ([ctypes.POINTER(ctypes.c_double), I, ctypes.POINTER(I)], S),
            "mlkv_profile_disable": ([], None),
            "mlkv_profile_launch_floor": ([I, I, I, ctypes.c_void_p,
                                           ctypes.POINTER(ctypes.c_double)], S),
            "mlkv_profile_read_bandwidth": ([ctypes.c_void_p, ctypes.c_size_t, I, ctypes.c_void_p,
                                             ctypes.POINTER(ctypes.c_double),
                                             ctypes.POINTER(ctypes.c_double)], S),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def _check(status: int):
    if status != MLKV_OK:
        raise MLKVError(status, lib().mlkv_last_error().decode())


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _dev_ptr(t: torch.Tensor, dtype, name: str) -> int:
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


# --------------------------------------------------------------------- map ---

class Map:
    """Layer -> KV-head map (owned by the library)."""

    def __init__(self, handle: int):
        self._h = ctypes.c_void_p(handle)

    @classmethod
    def uniform(cls, l: int, h: int, m: int, g: int) -> "Map":
        out = ctypes.c_void_p()
        _check(lib().mlkv_map_create_uniform(l, h, m, g, ctypes.byref(out)))
        return cls(out.value)

    @classmethod
    def from_tables(cls, kv_of, owner_of) -> "Map":
        kv_of = np.ascontiguousarray(kv_of, dtype=np.int32)
        owner_of = np.ascontiguousarray(owner_of, dtype=np.int32)
        l, h = kv_of.shape
        out = ctypes.c_void_p()
        _check(lib().mlkv_map_create(l, h, owner_of.size, kv_of.ctypes.data,
                                     owner_of.ctypes.data, ctypes.byref(out)))
        return cls(out.value)

    def __del__(self):
        if getattr(self, "_h", None) and self._h.value and _lib is not None:
            _lib.mlkv_map_destroy(self._h)
            self._h = ctypes.c_void_p()

    @property
    def handle(self):
        return self._h

    @property
    def l(self) -> int:
        return lib().mlkv_map_num_layers(self._h)

    @property
    def h(self) -> int:
        return lib().mlkv_map_num_q_heads(self._h)

    @property
    def n_kv(self) -> int:
        return lib().mlkv_map_num_kv_heads(self._h)

    def kv_head(self, layer: int, q_head: int) -> int:
        return lib().mlkv_map_kv_head(self._h, layer, q_head)

    def owner(self, kv: int) -> int:
        return lib().mlkv_map_owner_layer(self._h, kv)

    def kv_of(self) -> np.ndarray:
        return np.array([[self.kv_head(n, i) for i in range(self.h)] for n in range(self.l)],
                        dtype=np.int32)

    def owner_of(self) -> np.ndarray:
        return np.array([self.owner(k) for k in range(self.n_kv)], dtype=np.int32)

    def layer_kv_count(self, layer: int) -> int:
        return lib().mlkv_map_layer_kv_count(self._h, layer)

    def layer_owned(self, layer: int):
        """(first KV head, count) the layer appends; (-1, 0) if none."""
        return (lib().mlkv_map_layer_owned_begin(self._h, layer),
                lib().mlkv_map_layer_owned_count(self._h, layer))

    def cache_bytes(self, batch: int, capacity: int, head_dim: int) -> int:
        return lib().mlkv_cache_bytes(self._h, batch, capacity, head_dim)

    def workspace_bytes(self, batch: int, capacity: int, head_dim: int,
                        rotary_dims: int = 0) -> int:
        """mlkv_workspace_bytes, or mlkv_workspace_bytes_rope when rotary_dims > 0."""
        if rotary_dims:
            return lib().mlkv_workspace_bytes_rope(self._h, batch, capacity, head_dim, rotary_dims)
        return lib().mlkv_workspace_bytes(self._h, batch, capacity, head_dim)

    def plan(self, layer: int, batch: int, capacity: int, head_dim: int, max_len: int = 0):
        """(workgroups, max_parts) of mlkv_plan."""
        wg, mp = ctypes.c_int(), ctypes.c_int()
        _check(lib().mlkv_plan(self._h, layer, batch, capacity, head_dim, max_len,
                               ctypes.byref(wg), ctypes.byref(mp)))
        return wg.value, mp.value

    def plan_merge_kernel(self, layer: int, batch: int, capacity: int, head_dim: int,
                          max_len: int = 0) -> bool:
        """mlkv_plan_merge_kernel: whether a separate merge kernel follows the
        attention launch of that plan."""
        r = lib().mlkv_plan_merge_kernel(self._h, layer, batch, capacity, head_dim, max_len)
        if r < 0:
            raise ValueError("invalid plan arguments")
        return bool(r)


# ------------------------------------------------------------------- cache ---

class Cache:
    """KV cache planes in device memory (torch tensors, caller-owned).

    k: [n_kv][B][S][D] bf16 elements, each 32-token block of a sequence in
    the matrix-core operand order;  v: [n_kv][B][S/32][D][32] bf16
    (channel-major 32-token blocks).  The layout is the one documented in
    mlkv.h; write_rows / read_rows convert from and to plain token rows."""

    def __init__(self, k: torch.Tensor, v: torch.Tensor):
        n_kv, B, S, D = k.shape
        if tuple(v.shape) != (n_kv, B, S // V_BLOCK, D, V_BLOCK) or S % V_BLOCK:
            raise ValueError("value plane must be [n_kv][B][S/32][D][32] with S % 32 == 0")
        self.k, self.v = k, v
        self.n_kv, self.batch, self.capacity, self.head_dim = n_kv, B, S, D
        self._c = _Cache(_dev_ptr(k, torch.bfloat16, "cache.k"),
                         _dev_ptr(v, torch.bfloat16, "cache.v"), n_kv, B, S, D)

    @classmethod
    def empty(cls, n_kv: int, batch: int, capacity: int, head_dim: int, device="cuda") -> "Cache":
        k = torch.empty((n_kv, batch, capacity, head_dim), dtype=torch.bfloat16, device=device)
        v = torch.empty((n_kv, batch, capacity // V_BLOCK, head_dim, V_BLOCK),
                        dtype=torch.bfloat16, device=device)
        return cls(k, v)

    @property
    def struct(self):
        return ctypes.byref(self._c)

    def write_rows(self, k_rows: torch.Tensor, v_rows: torch.Tensor, kv_begin: int = 0,
                   stream=None):
        """mlkv_cache_write_rows: device rows [n][B][S][D] bf16 (plain row-major
        token rows) into the planes of KV heads kv_begin .. kv_begin + n - 1."""
        n = k_rows.shape[0]
        shape = (n, self.batch, self.capacity, self.head_dim)
        if tuple(k_rows.shape) != shape or tuple(v_rows.shape) != shape:
            raise ValueError(f"rows must be {shape}")
        _check(lib().mlkv_cache_write_rows(self.struct, kv_begin, n,
                                           _dev_ptr(k_rows, torch.bfloat16, "k_rows"),
                                           _dev_ptr(v_rows, torch.bfloat16, "v_rows"),
                                           _stream(stream)))

    def read_rows(self, kv_begin: int = 0, kv_count: int | None = None, stream=None):
        """mlkv_cache_read_rows: the planes of KV heads kv_begin .. +kv_count-1
        as device rows (k, v), each [kv_count][B][S][D] bf16."""
        n = self.n_kv - kv_begin if kv_count is None else kv_count
        shape = (n, self.batch, self.capacity, self.head_dim)
        k = torch.empty(shape, dtype=torch.bfloat16, device=self.k.device)
        v = torch.empty(shape, dtype=torch.bfloat16, device=self.k.device)
        _check(lib().mlkv_cache_read_rows(self.struct, kv_begin, n, _dev_ptr(k, torch.bfloat16, "k"),
                                          _dev_ptr(v, torch.bfloat16, "v"), _stream(stream)))
        return k, v

    def load_rows(self, k_rows: np.ndarray, v_rows: np.ndarray, kv_range=None):
        """Upload logical host rows ([n][B][S][D] bf16 bit patterns, uint16) for
        the KV heads kv_range (default: all) and write them into the planes
        on the device (mlkv_cache_write_rows)."""
        lo, hi = kv_range if kv_range is not None else (0, self.n_kv)
        assert k_rows.shape == (hi - lo, self.batch, self.capacity, self.head_dim)
        assert v_rows.shape == k_rows.shape
        dev = self.k.device
        self.write_rows(bf16_tensor(k_rows, dev), bf16_tensor(v_rows, dev), lo)


def bf16_tensor(a: np.ndarray, device=None) -> torch.Tensor:
    """uint16 bf16 bit patterns (numpy) -> torch bfloat16 tensor (bit exact)."""
    t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    return t if device is None else t.to(device)


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """torch bfloat16 tensor -> uint16 bit patterns (numpy, host)."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def workspace(map_: Map, batch: int, capacity: int, head_dim: int, device="cuda",
              stream=None, rotary_dims: int = 0) -> torch.Tensor:
    """Allocate and initialise (mlkv_workspace_init) a decode workspace (with
    room for the rotary table of mlkv_decode_step_rope when rotary_dims > 0)."""
    n = map_.workspace_bytes(batch, capacity, head_dim, rotary_dims)
    ws = torch.empty(max(n, 16), dtype=torch.uint8, device=device)
    _check(lib().mlkv_workspace_init(ws.data_ptr(), ws.numel(), _stream(stream)))
    return ws


# --------------------------------------------------------------- entry points

def cache_append(layer: int, map_: Map, cache: Cache, k_new: torch.Tensor, v_new: torch.Tensor,
                 positions: torch.Tensor, row_stride: int | None = None, stream=None):
    """mlkv_cache_append: k_new/v_new [B][owned][D] (or rows of `row_stride` elements)."""
    if row_stride is None:
        row_stride = k_new[0].numel() if k_new.dim() > 1 else k_new.numel()
    _check(lib().mlkv_cache_append(layer, map_.handle, cache.struct,
                                   _dev_ptr(k_new, torch.bfloat16, "k_new"),
                                   _dev_ptr(v_new, torch.bfloat16, "v_new"), row_stride,
                                   _dev_ptr(positions, torch.int32, "positions"), _stream(stream)))


def decode_attention(layer: int, q: torch.Tensor, cache: Cache, map_: Map, seq_lens: torch.Tensor,
                     out: torch.Tensor, max_len_hint: int = 0, ws: torch.Tensor | None = None,
                     stream=None):
    """mlkv_decode_attention: q [B][h][D] bf16 -> out [B][h][D] (fp32 or bf16)."""
    out_dt = OUT_BF16 if out.dtype == torch.bfloat16 else OUT_F32
    if out.dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("out must be float32 or bfloat16")
    ws_ptr, ws_n = (ws.data_ptr(), ws.numel() * ws.element_size()) if ws is not None else (None, 0)
    _check(lib().mlkv_decode_attention(layer, _dev_ptr(q, torch.bfloat16, "q"), cache.struct,
                                       map_.handle, _dev_ptr(seq_lens, torch.int32, "seq_lens"),
                                       _dev_ptr(out, out.dtype, "out"), out_dt, max_len_hint,
                                       ws_ptr, ws_n, _stream(stream)))


def decode_step(q_all: torch.Tensor, k_new_all: torch.Tensor, v_new_all: torch.Tensor,
                cache: Cache, map_: Map, ctx_lens: torch.Tensor, out_all: torch.Tensor,
                max_len_hint: int = 0, ws: torch.Tensor | None = None, stream=None,
                rotary_dims: int = 0, rotary_base: float = 10000.0):
    """mlkv_decode_step over all layers: q_all [l][B][h][D], k/v_new_all [B][n_kv][D].
    rotary_dims > 0 calls mlkv_decode_step_rope: the newest token's queries
    and keys are rotated at position ctx_lens[b] inside the step (q_all and
    k_new_all are not written); ws must then come from
    workspace(..., rotary_dims=rotary_dims)."""
    out_dt = OUT_BF16 if out_all.dtype == torch.bfloat16 else OUT_F32
    if out_all.dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("out_all must be float32 or bfloat16")
    ws_ptr, ws_n = (ws.data_ptr(), ws.numel() * ws.element_size()) if ws is not None else (None, 0)
    args = (_dev_ptr(q_all, torch.bfloat16, "q_all"),
            _dev_ptr(k_new_all, torch.bfloat16, "k_new_all"),
            _dev_ptr(v_new_all, torch.bfloat16, "v_new_all"), cache.struct, map_.handle,
            _dev_ptr(ctx_lens, torch.int32, "ctx_lens"))
    tail = (_dev_ptr(out_all, out_all.dtype, "out_all"), out_dt, max_len_hint, ws_ptr, ws_n,
            _stream(stream))
    if rotary_dims:
        _check(lib().mlkv_decode_step_rope(*args, rotary_dims, float(rotary_base), *tail))
    else:
        _check(lib().mlkv_decode_step(*args, *tail))


def cache_append_rows(layer: int, map_: Map, cache: Cache, k_new: torch.Tensor,
                      v_new: torch.Tensor, ctx_lens: torch.Tensor, T: int,
                      row_stride: int | None = None, stream=None):
    """mlkv_cache_append_rows: k_new/v_new [B][T][owned][D] (or rows of
    `row_stride` elements), stored at slots ctx_lens[b] + t."""
    if row_stride is None:
        row_stride = k_new[0, 0].numel()
    _check(lib().mlkv_cache_append_rows(layer, map_.handle, cache.struct,
                                        _dev_ptr(k_new, torch.bfloat16, "k_new"),
                                        _dev_ptr(v_new, torch.bfloat16, "v_new"), T, row_stride,
                                        _dev_ptr(ctx_lens, torch.int32, "ctx_lens"),
                                        _stream(stream)))


def prefill_attention(layer: int, q: torch.Tensor, cache: Cache, map_: Map,
                      ctx_lens: torch.Tensor, out: torch.Tensor, stream=None):
    """mlkv_prefill_attention: q [B][T][h][D] bf16 -> out [B][T][h][D] (fp32
    or bf16); token t of sequence b attends positions 0 .. ctx_lens[b] + t."""
    if out.dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("out must be float32 or bfloat16")
    out_dt = OUT_BF16 if out.dtype == torch.bfloat16 else OUT_F32
    _check(lib().mlkv_prefill_attention(layer, _dev_ptr(q, torch.bfloat16, "q"), cache.struct,
                                        map_.handle, _dev_ptr(ctx_lens, torch.int32, "ctx_lens"),
                                        q.shape[1], _dev_ptr(out, out.dtype, "out"), out_dt,
                                        _stream(stream)))


def prefill_step(q_all: torch.Tensor, k_new_all: torch.Tensor, v_new_all: torch.Tensor,
                 cache: Cache, map_: Map, ctx_lens: torch.Tensor, out_all: torch.Tensor,
                 stream=None):
    """mlkv_prefill_step: q_all [l][B][T][h][D], k/v_new_all [B][T][n_kv][D]
    -> out_all [l][B][T][h][D]; owners store their rows, every layer attends
    causally."""
    if out_all.dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("out_all must be float32 or bfloat16")
    out_dt = OUT_BF16 if out_all.dtype == torch.bfloat16 else OUT_F32
    _check(lib().mlkv_prefill_step(_dev_ptr(q_all, torch.bfloat16, "q_all"),
                                   _dev_ptr(k_new_all, torch.bfloat16, "k_new_all"),
                                   _dev_ptr(v_new_all, torch.bfloat16, "v_new_all"), cache.struct,
                                   map_.handle, _dev_ptr(ctx_lens, torch.int32, "ctx_lens"),
                                   q_all.shape[2], _dev_ptr(out_all, out_all.dtype, "out_all"),
                                   out_dt, _stream(stream)))


# ---------------------------------------------------------------- model ---

LAYER_WEIGHT_NAMES = ("ln1_w", "ln1_b", "ln2_w", "ln2_b", "w_q", "b_q", "w_k", "b_k", "w_v", "b_v",
                      "w_o", "b_o", "w_fc1", "b_fc1", "w_fc2", "b_fc2")


class _LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in LAYER_WEIGHT_NAMES]


class Model:
    """mlkv_model: GPT-NeoX layers around the MLKV attention.  `layers` is a
    list (one per layer) of dicts name -> bf16 device tensor (None for the
    key/value weights of a layer owning no KV head); the tensors are kept
    alive by this object."""

    def __init__(self, map_: Map, d_model: int, d_ff: int, head_dim: int, layers,
                 rotary_dims: int = 16, rotary_base: float = 10000.0, ln_eps: float = 1e-5):
        self.map, self._layers = map_, layers
        arr = (_LayerWeights * len(layers))()
        for i, lw in enumerate(layers):
            for n in LAYER_WEIGHT_NAMES:
                t = lw.get(n)
                setattr(arr[i], n, None if t is None else _dev_ptr(t, torch.bfloat16, n))
        self._arr = arr
        out = ctypes.c_void_p()
        _check(lib().mlkv_model_create(map_.handle, d_model, d_ff, head_dim, rotary_dims,
                                       float(rotary_base), float(ln_eps), arr,
                                       ctypes.byref(out)))
        self._h = out

    def __del__(self):
        if getattr(self, "_h", None) and self._h.value and _lib is not None:
            _lib.mlkv_model_destroy(self._h)
            self._h = ctypes.c_void_p()

    def fused_path(self, batch: int) -> bool:
        """mlkv_model_fused_path: whether `batch` sequences run on the fused kernels."""
        return bool(lib().mlkv_model_fused_path(self._h, batch))

    def workspace(self, batch: int, capacity: int, device="cuda", stream=None) -> torch.Tensor:
        n = lib().mlkv_model_workspace_bytes(self._h, batch, capacity)
        if n == 0:
            raise ValueError("invalid model workspace arguments")
        ws = torch.empty(n, dtype=torch.uint8, device=device)
        _check(lib().mlkv_workspace_init(ws.data_ptr(), n, _stream(stream)))
        return ws

    def decode_step(self, x: torch.Tensor, cache: Cache, ctx_lens: torch.Tensor,
                    ws: torch.Tensor, max_len_hint: int = 0, stream=None):
        """mlkv_model_decode_step: x [B][d_model] fp32, updated in place."""
        _check(lib().mlkv_model_decode_step(self._h, _dev_ptr(x, torch.float32, "x"), cache.struct,
                                            _dev_ptr(ctx_lens, torch.int32, "ctx_lens"),
                                            max_len_hint, ws.data_ptr(),
                                            ws.numel() * ws.element_size(), _stream(stream)))


# ------------------------------------------------------------------ timing ---

def profile_enable(max_launches: int):
    """Bracket the next attention kernels with HIP events (mlkv_profile_enable)."""
    _check(lib().mlkv_profile_enable(max_launches))


def profile_read():
    """(launches, total_ms, min_ms, max_ms) of the timed attention kernels."""
    n = ctypes.c_int()
    tot, lo, hi = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    _check(lib().mlkv_profile_read(ctypes.byref(n), ctypes.byref(tot), ctypes.byref(lo),
                                   ctypes.byref(hi)))
    return n.value, tot.value, lo.value, hi.value


def profile_durations(capacity: int) -> np.ndarray:
    """Per-launch durations (ms) of the timed attention kernels, in order."""
    buf = (ctypes.c_double * max(capacity, 1))()
    n = ctypes.c_int()
    _check(lib().mlkv_profile_durations(buf, capacity, ctypes.byref(n)))
    return np.array(buf[:n.value], dtype=np.float64)


def profile_disable():
    lib().mlkv_profile_disable()


def profile_read_bandwidth(buffer: torch.Tensor, reps: int = 10, stream=None):
    """(median, best) GB/s of a plain streaming read of `buffer`
    (mlkv_profile_read_bandwidth)."""
    med, best = ctypes.c_double(), ctypes.c_double()
    _check(lib().mlkv_profile_read_bandwidth(buffer.data_ptr(), buffer.numel() * buffer.element_size(),
                                             reps, _stream(stream), ctypes.byref(med),
                                             ctypes.byref(best)))
    return med.value, best.value


def profile_launch_floor(workgroups: int, threads: int = 256, reps: int = 100,
                         stream=None) -> float:
    """Median event-pair duration (ms) of an empty kernel of the given shape
    (mlkv_profile_launch_floor)."""
    ms = ctypes.c_double()
    _check(lib().mlkv_profile_launch_floor(workgroups, threads, reps, _stream(stream),
                                           ctypes.byref(ms)))
    return ms.value
