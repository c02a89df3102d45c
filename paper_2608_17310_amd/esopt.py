"""ctypes binding of libesopt.so (the C ABI in include/esopt.h).

Argument marshalling only: every step of the ES parameter path runs in the HIP
kernels of the library.  PyTorch supplies device memory and the current HIP
stream.  The library is loaded on first use; if it has not been built the
call raises (there is no fallback).

    plan = Plan([w0, w1, ...])           # bf16, contiguous, on the current device
    plan.perturb(seed, sign, sigma)      # theta += sign sigma eps(seed)
    plan.restore(seed, sign, sigma)      # theta -= sign sigma eps(seed)
    plan.swap(seed_a, sign_a, seed_b, sign_b, sigma)   # restore a + perturb b, one pass
    plan.update(seeds, signs, rewards, alpha)   # fused z-score + N-member update
    plan.checksum()                      # 64-bit checksum of the parameters
"""

import ctypes
import os

import torch

LIB_NAME = "libesopt.so"
LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), LIB_NAME)

ES_OK = 0
ES_ERR_INVALID_ARG = -1
ES_ERR_ALIGN = -2
ES_ERR_HIP = -3
ES_ERR_DEVICE = -4
ES_ERR_NOMEM = -5
ES_MAX_MEMBERS = 1024
ES_UPDATE_DIV_SIGMA = 1
ES_REWARDS_ARE_WEIGHTS = 2
ES_UPDATE_STOCHASTIC_ROUND = 4
ES_UPDATE_MASTER = 8

# Every symbol the header declares, with (restype, argtypes).
_u32, _u64, _i32, _f32, _f64 = (ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int32,
                                ctypes.c_float, ctypes.c_double)
_vp = ctypes.c_void_p


class EsTensor(ctypes.Structure):
    _fields_ = [("data", _vp), ("numel", _u64), ("tensor_id", _u32), ("offset8", _u32)]


class EsBlock(ctypes.Structure):
    _fields_ = [("data", _vp), ("rows", _u64), ("cols", _u64), ("row_len", _u64),
                ("row0", _u64), ("col0", _u64), ("tensor_id", _u32), ("reserved", _u32)]


class EsQTensor(ctypes.Structure):
    _fields_ = [("data", _vp), ("scales", _vp), ("numel", _u64), ("row", _u32),
                ("tensor_id", _u32)]


class EsQBlock(ctypes.Structure):
    _fields_ = [("data", _vp), ("scales", _vp), ("rows", _u64), ("cols", _u64),
                ("row_len", _u64), ("row0", _u64), ("col0", _u64), ("row", _u32),
                ("tensor_id", _u32)]


class EsTileInfo(ctypes.Structure):
    _fields_ = [("elem0", _u64), ("end", _u64), ("full", _u32), ("aligned16", _u32)]


class EsUpdateOpts(ctypes.Structure):
    _fields_ = [("alpha", _f32), ("sigma", _f32), ("zscore_eps", _f32), ("flags", _u32),
                ("round_seed", _u64)]


SIGNATURES = {
    "es_plan_create": (ctypes.c_int, [ctypes.POINTER(EsTensor), _u32, ctypes.POINTER(_vp)]),
    "es_plan_create_blocks": (ctypes.c_int, [ctypes.POINTER(EsBlock), _u32,
                                             ctypes.POINTER(_vp)]),
    "es_plan_destroy": (ctypes.c_int, [_vp]),
    "es_plan_set_master": (ctypes.c_int, [_vp, ctypes.POINTER(_vp), _u32]),
    "es_perturb_master": (ctypes.c_int, [_vp, _u64, _i32, _f32, _vp]),
    "es_plan_numel": (_u64, [_vp]),
    "es_plan_tiles": (_u64, [_vp]),
    "es_plan_device_bytes": (_u64, [_vp]),
    "es_perturb": (ctypes.c_int, [_vp, _u64, _i32, _f32, _vp]),
    "es_restore": (ctypes.c_int, [_vp, _u64, _i32, _f32, _vp]),
    "es_swap": (ctypes.c_int, [_vp, _u64, _i32, _f32, _u64, _i32, _f32, _vp]),
    "es_stream_pass": (ctypes.c_int, [_vp, _vp]),
    "es_plan_checksum": (ctypes.c_int, [_vp, _vp, _vp]),
    "es_hbm_calibrate": (ctypes.c_int, [_vp, _u64, _i32, _vp, _vp]),
    "es_zscore": (ctypes.c_int, [_vp, _u32, _f32, _vp, _vp, _vp]),
    "es_update": (ctypes.c_int, [_vp, ctypes.POINTER(_u64), ctypes.POINTER(_i32), _vp, _u32,
                                 ctypes.POINTER(EsUpdateOpts), _vp, _vp, _vp]),
    "es_update_noalloc": (ctypes.c_int, [_vp, ctypes.POINTER(_u64), ctypes.POINTER(_i32), _vp,
                                         _u32, ctypes.POINTER(EsUpdateOpts), _vp, _vp, _vp]),
    "es_restore_update": (ctypes.c_int, [_vp, _u64, _i32, _f32, ctypes.POINTER(_u64),
                                         ctypes.POINTER(_i32), _vp, _u32,
                                         ctypes.POINTER(EsUpdateOpts), _vp, _vp, _vp]),
    "es_qplan_create": (ctypes.c_int, [ctypes.POINTER(EsQTensor), _u32, ctypes.POINTER(_vp)]),
    "es_qplan_create_format": (ctypes.c_int, [ctypes.POINTER(EsQTensor), _u32, _u32,
                                              ctypes.POINTER(_vp)]),
    "es_qplan_create_shards": (ctypes.c_int, [ctypes.POINTER(EsQTensor),
                                              ctypes.POINTER(ctypes.c_uint64), _u32, _u32,
                                              ctypes.POINTER(_vp)]),
    "es_qplan_create_blocks": (ctypes.c_int, [ctypes.POINTER(EsQBlock), _u32, _u32,
                                              ctypes.POINTER(_vp)]),
    "es_qswap": (ctypes.c_int, [_vp, _u64, _i32, _f32, _u64, _i32, _f32, _vp]),
    "es_qplan_destroy": (ctypes.c_int, [_vp]),
    "es_qplan_numel": (_u64, [_vp]),
    "es_qplan_device_bytes": (_u64, [_vp]),
    "es_qplan_checksum": (ctypes.c_int, [_vp, _vp, _vp]),
    "es_qperturb": (ctypes.c_int, [_vp, _u64, _i32, _f32, _vp]),
    "es_qrestore": (ctypes.c_int, [_vp, _u64, _i32, _f32, _vp]),
    "es_qupdate": (ctypes.c_int, [_vp, ctypes.POINTER(_u64), ctypes.POINTER(_i32), _vp, _u32,
                                  ctypes.POINTER(EsUpdateOpts), _vp, _vp, _vp]),
    "es_sigma_cosine": (_f64, [_f64, _f64, _u32, _u32]),
    "es_philox_words": (ctypes.c_int, [_u64, _u32, _u32, _u64, _u64, _vp, _vp]),
    "es_normals": (ctypes.c_int, [_u64, _u32, _u64, _u64, _vp, _vp]),
    "es_tile_layout": (ctypes.c_int, [_u64, _u64, _u32, ctypes.POINTER(EsTileInfo), _u64,
                                      ctypes.POINTER(_u64)]),
    "es_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "es_last_error": (ctypes.c_char_p, []),
}

_lib = None


class EsError(RuntimeError):
    def __init__(self, code, what, detail):
        super().__init__(f"{what}: {name_of(code)}: {detail}")
        self.code = code


def load():
    """Load libesopt.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; "
                f"g.build()'` (hipcc, gfx950); there is no CPU fallback")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def name_of(code):
    return load().es_strerror(code).decode()


def last_error():
    return load().es_last_error().decode()


def _check(rc, what):
    if rc != ES_OK:
        raise EsError(rc, what, last_error())


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _u64_arg(x, what):
    """An integer argument of a uint64_t parameter, range-checked (ctypes
    would wrap a negative or oversized value silently)."""
    v = int(x)
    if not 0 <= v < (1 << 64):
        raise ValueError(f"{what} must be in [0, 2^64), got {v}")
    return v


def _u32_arg(x, what):
    v = int(x)
    if not 0 <= v < (1 << 32):
        raise ValueError(f"{what} must be in [0, 2^32), got {v}")
    return v


def _dev_ptr(t, dtype, what):
    """Pointer of a contiguous tensor the device can read: on the GPU, or in
    pinned (page-locked, device-mapped) host memory."""
    if t is None:
        return None
    if not (t.is_cuda or t.is_pinned()) or t.dtype != dtype or not t.is_contiguous():
        raise ValueError(f"{what} must be a contiguous {dtype} tensor on the GPU or pinned")
    return ctypes.c_void_p(t.data_ptr())


class Block(tuple):
    """One block of es_plan_create_blocks: Block(tensor, tensor_id, row_len,
    row0=0, col0=0), the whole tensor's rows row0.. and columns col0.. of a
    row-major tensor with row_len columns, stored as `tensor` ([rows, cols]
    contiguous, or 1-D for one row)."""

    def __new__(cls, tensor, tensor_id, row_len, row0=0, col0=0):
        return super().__new__(cls, (tensor, tensor_id, row_len, row0, col0))


class Plan:
    """A list of bf16 parameter tensors prepared for single-launch passes.

    tensor_ids defaults to the list index.  offsets (multiples of 8, default
    0) place shards: element i of tensors[k] carries the noise of element
    offsets[k] + i of the whole tensor tensor_ids[k].  Plan(blocks=[Block...])
    plans rectangular blocks of row-major tensors instead (column or
    row-and-column shards; es_plan_create_blocks).  The plan holds
    references to the tensors so their storage stays alive and in place
    while it exists.
    """

    def __init__(self, tensors=None, tensor_ids=None, offsets=None, blocks=None):
        if blocks is not None:
            if tensors is not None or tensor_ids is not None or offsets is not None:
                raise ValueError("give either tensors or blocks")
            self._init_blocks(list(blocks))
            return
        tensors = list(tensors if tensors is not None else [])
        if not tensors:
            raise ValueError("empty tensor list")
        ids = (list(range(len(tensors))) if tensor_ids is None
               else [_u32_arg(i, "tensor_id") for i in tensor_ids])
        if len(ids) != len(tensors):
            raise ValueError("tensor_ids must match tensors")
        offs = [0] * len(tensors) if offsets is None else [_offset8(o) for o in offsets]
        if len(offs) != len(tensors):
            raise ValueError("offsets must match tensors")
        arr = (EsTensor * len(tensors))()
        for i, (t, tid, o8) in enumerate(zip(tensors, ids, offs)):
            if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous():
                raise ValueError(f"tensor {i} must be a contiguous bf16 CUDA tensor")
            arr[i] = EsTensor(t.data_ptr() if t.numel() else None, t.numel(), tid, o8)
        self._tensors = tensors
        self.tensor_ids = ids
        self.device = tensors[0].device
        handle = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            _check(load().es_plan_create(arr, len(tensors), ctypes.byref(handle)), "es_plan_create")
        self._h = handle

    def _init_blocks(self, blocks):
        """es_plan_create_blocks.  Each block is (tensor, tensor_id, row_len,
        row0, col0): `tensor` a contiguous bf16 CUDA tensor of shape
        [rows, cols] (1-D: one row) holding the whole tensor's rows
        row0.. and columns col0.. of a row-major tensor with row_len columns
        (Block names the fields)."""
        if not blocks:
            raise ValueError("empty block list")
        arr = (EsBlock * len(blocks))()
        tensors, ids = [], []
        for i, b in enumerate(blocks):
            t, tid, row_len, row0, col0 = b
            if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous():
                raise ValueError(f"block {i} must be a contiguous bf16 CUDA tensor")
            if t.dim() == 1:
                rows, cols = 1, t.numel()
            elif t.dim() == 2:
                rows, cols = t.shape
            else:
                raise ValueError(f"block {i} must be 1-D or 2-D")
            arr[i] = EsBlock(t.data_ptr() if t.numel() else None, rows, cols,
                             _u64_arg(row_len, "row_len"), _u64_arg(row0, "row0"),
                             _u64_arg(col0, "col0"), _u32_arg(tid, "tensor_id"), 0)
            tensors.append(t)
            ids.append(int(tid))
        self._tensors = tensors
        self.tensor_ids = ids
        self.device = tensors[0].device
        handle = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            _check(load().es_plan_create_blocks(arr, len(blocks), ctypes.byref(handle)),
                   "es_plan_create_blocks")
        self._h = handle

    @property
    def handle(self):
        if self._h is None:
            raise RuntimeError("plan is closed")
        return self._h

    @property
    def numel(self):
        return int(load().es_plan_numel(self.handle))

    @property
    def tiles(self):
        return int(load().es_plan_tiles(self.handle))

    @property
    def device_bytes(self):
        """Device memory the plan allocates for itself (table and scratch)."""
        return int(load().es_plan_device_bytes(self.handle))

    @property
    def tensors(self):
        return list(self._tensors)

    def perturb(self, seed, sign, sigma, stream=None):
        _check(load().es_perturb(self.handle, _u64_arg(seed, "seed"), int(sign), float(sigma),
                                 _stream(stream)), "es_perturb")

    def restore(self, seed, sign, sigma, stream=None):
        _check(load().es_restore(self.handle, _u64_arg(seed, "seed"), int(sign), float(sigma),
                                 _stream(stream)), "es_restore")

    def stream_pass(self, stream=None):
        """Read every parameter and write it back unchanged over es_perturb's
        tiles, with no arithmetic (the in-place streaming ceiling)."""
        _check(load().es_stream_pass(self.handle, _stream(stream)), "es_stream_pass")

    def checksum(self, out=None, stream=None):
        """64-bit checksum of the parameters (es_plan_checksum).  Without
        `out`, returns it as a Python int (synchronising); with `out`, a
        one-element int64 tensor on the plan's device, the value (its bits)
        is left there, stream-ordered, and `out` is returned."""
        return _call_checksum(load().es_plan_checksum, "es_plan_checksum", self, out, stream)

    def swap(self, seed_from, sign_from, seed_to, sign_to, sigma, sigma_to=None, stream=None):
        """Revert member `from` and apply member `to` in one pass: the same
        bits as restore(from) followed by perturb(to)."""
        sigma_to = sigma if sigma_to is None else sigma_to
        _check(load().es_swap(self.handle, _u64_arg(seed_from, "seed_from"), int(sign_from),
                              float(sigma), _u64_arg(seed_to, "seed_to"), int(sign_to),
                              float(sigma_to), _stream(stream)), "es_swap")

    def update(self, seeds, signs, rewards, alpha, sigma=0.0, zscore_eps=1e-8, flags=0,
               z_out=None, status_out=None, stream=None, round_seed=0):
        """Fused update; rewards is a float32 CUDA tensor of len(seeds).
        round_seed keys the draws of ES_UPDATE_STOCHASTIC_ROUND."""
        _call_update(load().es_update, "es_update", self.handle, seeds, signs, rewards, alpha,
                     sigma, zscore_eps, flags, z_out, status_out, stream, round_seed)

    def restore_update(self, restore_seed, restore_sign, restore_sigma, seeds, signs, rewards,
                       alpha, sigma=0.0, zscore_eps=1e-8, flags=0, z_out=None, status_out=None,
                       stream=None, round_seed=0):
        """restore(restore_seed, restore_sign, restore_sigma) followed by
        update(seeds, ...), the same bits in one pass (es_restore_update);
        the restored seed must be one of `seeds`."""
        rs, rsign, rsig = _u64_arg(restore_seed, "restore_seed"), int(restore_sign), \
            float(restore_sigma)

        def fn(handle, *rest):
            return load().es_restore_update(handle, rs, rsign, rsig, *rest)
        _call_update(fn, "es_restore_update", self.handle, seeds, signs, rewards, alpha, sigma,
                     zscore_eps, flags, z_out, status_out, stream, round_seed)

    def set_master(self, masters):
        """Attach binary32 master copies (es_plan_set_master): masters[i] a
        contiguous float32 CUDA tensor with the element count of the plan's
        tensor (or block) i, 16-byte aligned.  Updates with
        flags=ES_UPDATE_MASTER then accumulate into them and rewrite the bf16
        tensors as their nearest-even rounding.  None detaches them."""
        if masters is None:
            _check(load().es_plan_set_master(self.handle, None, 0), "es_plan_set_master")
            self._masters = None
            return
        masters = list(masters)
        if len(masters) != len(self._tensors):
            raise ValueError(f"{len(masters)} masters for {len(self._tensors)} tensors")
        arr = (_vp * len(masters))()
        for i, (m, t) in enumerate(zip(masters, self._tensors)):
            if m.dtype != torch.float32 or not m.is_cuda or not m.is_contiguous():
                raise ValueError(f"master {i} must be a contiguous float32 CUDA tensor")
            if m.numel() != t.numel():
                raise ValueError(f"master {i} has {m.numel()} elements, its tensor {t.numel()}")
            arr[i] = m.data_ptr() if m.numel() else None
        with torch.cuda.device(self.device):
            _check(load().es_plan_set_master(self.handle, arr, len(masters)),
                   "es_plan_set_master")
        self._masters = masters

    @property
    def has_master(self):
        return getattr(self, "_masters", None) is not None

    def perturb_master(self, seed, sign, sigma, stream=None):
        """bf16 values = RNE(master + sign sigma eps(seed)) (es_perturb_master):
        a member applied from the masters, which stay unchanged; sigma 0
        refreshes the bf16 values from the masters."""
        _check(load().es_perturb_master(self.handle, _u64_arg(seed, "seed"), int(sign),
                                        float(sigma), _stream(stream)), "es_perturb_master")

    def update_noalloc(self, seeds, signs, rewards, alpha, sigma=0.0, zscore_eps=1e-8, flags=0,
                       z_out=None, status_out=None, stream=None, round_seed=0):
        """update() through es_update_noalloc: the member tables in the
        library's static device array (for callers that cannot allocate)."""
        _call_update(load().es_update_noalloc, "es_update_noalloc", self.handle, seeds, signs,
                     rewards, alpha, sigma, zscore_eps, flags, z_out, status_out, stream,
                     round_seed)

    def close(self):
        if self._h is not None:
            _check(load().es_plan_destroy(self._h), "es_plan_destroy")
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def _call_checksum(fn, what, plan, out, stream):
    ret = out is None
    if ret:
        out = torch.empty(1, dtype=torch.int64, device=plan.device)
    elif out.numel() != 1 or out.device != plan.device:
        raise ValueError("out must be a one-element tensor on the plan's device")
    _check(fn(plan.handle, _dev_ptr(out, torch.int64, "out"), _stream(stream)), what)
    if not ret:
        return out
    if stream is not None:
        torch.cuda.synchronize(plan.device)
    return int(out.item()) & ((1 << 64) - 1)


def _call_update(fn, what, handle, seeds, signs, rewards, alpha, sigma, zscore_eps, flags,
                 z_out, status_out, stream, round_seed):
    n = len(seeds)
    if len(signs) != n:
        raise ValueError("seeds and signs differ in length")
    if rewards.numel() != n:
        raise ValueError("rewards must have one entry per member")
    c_seeds = (_u64 * max(n, 1))(*[_u64_arg(s, "seed") for s in seeds])
    c_signs = (_i32 * max(n, 1))(*[int(s) for s in signs])
    opts = EsUpdateOpts(float(alpha), float(sigma), float(zscore_eps), _u32_arg(flags, "flags"),
                        _u64_arg(round_seed, "round_seed"))
    _check(fn(handle, c_seeds, c_signs, _dev_ptr(rewards, torch.float32, "rewards"), n,
              ctypes.byref(opts), _dev_ptr(z_out, torch.float32, "z_out"),
              _dev_ptr(status_out, torch.int32, "status_out"), _stream(stream)), what)


QFORMAT_INT8, QFORMAT_E4M3 = 0, 1
_QFORMATS = {"int8": QFORMAT_INT8, "e4m3": QFORMAT_E4M3}


class QBlock(tuple):
    """One block of es_qplan_create_blocks: QBlock(codes, scales, row,
    tensor_id, row_len, row0=0, col0=0), the whole tensor's rows row0.. and
    columns col0.. of a row-major quantized tensor with row_len codes per row,
    stored as `codes` ([rows, cols] contiguous, or 1-D for one row), with the
    block's own scales, one per `row` codes in its storage order."""

    def __new__(cls, codes, scales, row, tensor_id, row_len, row0=0, col0=0):
        return super().__new__(cls, (codes, scales, row, tensor_id, row_len, row0, col0))


class QPlan:
    """A list of quantized parameter tensors with binary32 scales (theta =
    s v(c), one scale per `row` consecutive codes, row a multiple of 8, 0 for
    one scale per tensor), prepared for single-launch passes.  format "int8":
    int8 codes, v(c) = c; format "e4m3": fp8 E4M3 codes (torch.float8_e4m3fn,
    or their bytes as torch.uint8).  offsets places shards: codes[k] holds
    elements offsets[k] .. of its whole tensor (a multiple of 16, and of the
    row length when rows[k] > 0; scales[k] are the shard's own rows of
    scales), as es_qplan_create_shards.  QPlan(blocks=[QBlock...]) plans
    rectangular blocks of row-major tensors instead (column or
    row-and-column shards; es_qplan_create_blocks).  The plan keeps
    references to the codes and scales."""

    def __init__(self, codes=None, scales=None, rows=None, tensor_ids=None, format="int8",
                 offsets=None, blocks=None):
        if format not in _QFORMATS:
            raise ValueError(f"format must be one of {sorted(_QFORMATS)}")
        self.format = format
        code_dtypes = ((torch.int8,) if format == "int8"
                       else (torch.float8_e4m3fn, torch.uint8))
        if blocks is not None:
            if any(a is not None for a in (codes, scales, rows, tensor_ids, offsets)):
                raise ValueError("give either codes, scales and rows, or blocks")
            self._init_blocks(list(blocks), code_dtypes)
            return
        if codes is None or scales is None or rows is None:
            raise ValueError("codes, scales and rows are required")
        codes, scales, rows = list(codes), list(scales), [int(r) for r in rows]
        if not codes or len(scales) != len(codes) or len(rows) != len(codes):
            raise ValueError("codes, scales and rows must be non-empty and of equal length")
        ids = (list(range(len(codes))) if tensor_ids is None
               else [_u32_arg(i, "tensor_id") for i in tensor_ids])
        if len(ids) != len(codes):
            raise ValueError("tensor_ids must match tensors")
        elem0 = None
        if offsets is not None:
            offs = [_u64_arg(o, "offset") for o in offsets]
            if len(offs) != len(codes):
                raise ValueError("offsets must match tensors")
            elem0 = (ctypes.c_uint64 * len(offs))(*offs)
        arr = (EsQTensor * len(codes))()
        for i, (q, sc, row, tid) in enumerate(zip(codes, scales, rows, ids)):
            if q.dtype not in code_dtypes or not q.is_cuda or not q.is_contiguous():
                raise ValueError(f"codes {i} must be a contiguous CUDA tensor of "
                                 f"{' or '.join(str(d) for d in code_dtypes)}")
            if sc.dtype != torch.float32 or not sc.is_cuda or not sc.is_contiguous():
                raise ValueError(f"scales {i} must be a contiguous float32 CUDA tensor")
            need = 1 if row == 0 else -(-q.numel() // row)
            if q.numel() and sc.numel() < need:
                raise ValueError(f"scales {i} has {sc.numel()} entries, needs {need}")
            arr[i] = EsQTensor(q.data_ptr() if q.numel() else None,
                               sc.data_ptr() if q.numel() else None, q.numel(), row, tid)
        self._keep = (codes, scales)
        self.tensor_ids = ids
        self.device = codes[0].device
        handle = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            _check(load().es_qplan_create_shards(arr, elem0, len(codes), _QFORMATS[format],
                                                 ctypes.byref(handle)), "es_qplan_create")
        self._h = handle

    def _init_blocks(self, blocks, code_dtypes):
        if not blocks:
            raise ValueError("empty block list")
        arr = (EsQBlock * len(blocks))()
        codes, scales, ids = [], [], []
        for i, (q, sc, row, tid, row_len, row0, col0) in enumerate(blocks):
            if q.dtype not in code_dtypes or not q.is_cuda or not q.is_contiguous():
                raise ValueError(f"block {i} must be a contiguous CUDA tensor of "
                                 f"{' or '.join(str(d) for d in code_dtypes)}")
            if q.dim() == 1:
                n_rows, n_cols = 1, q.numel()
            elif q.dim() == 2:
                n_rows, n_cols = q.shape
            else:
                raise ValueError(f"block {i} must be 1-D or 2-D")
            if sc.dtype != torch.float32 or not sc.is_cuda or not sc.is_contiguous():
                raise ValueError(f"scales {i} must be a contiguous float32 CUDA tensor")
            row = int(row)
            need = 1 if row == 0 else -(-q.numel() // row)
            if q.numel() and sc.numel() < need:
                raise ValueError(f"scales {i} has {sc.numel()} entries, needs {need}")
            arr[i] = EsQBlock(q.data_ptr() if q.numel() else None,
                              sc.data_ptr() if q.numel() else None, n_rows, n_cols,
                              _u64_arg(row_len, "row_len"), _u64_arg(row0, "row0"),
                              _u64_arg(col0, "col0"), _u32_arg(row, "row"),
                              _u32_arg(tid, "tensor_id"))
            codes.append(q)
            scales.append(sc)
            ids.append(int(tid))
        self._keep = (codes, scales)
        self.tensor_ids = ids
        self.device = codes[0].device
        handle = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            _check(load().es_qplan_create_blocks(arr, len(blocks), _QFORMATS[self.format],
                                                 ctypes.byref(handle)), "es_qplan_create_blocks")
        self._h = handle

    @property
    def handle(self):
        if self._h is None:
            raise RuntimeError("plan is closed")
        return self._h

    @property
    def numel(self):
        return int(load().es_qplan_numel(self.handle))

    @property
    def device_bytes(self):
        """Device memory the plan allocates for itself (table and scratch)."""
        return int(load().es_qplan_device_bytes(self.handle))

    def perturb(self, seed, sign, sigma, stream=None):
        _check(load().es_qperturb(self.handle, _u64_arg(seed, "seed"), int(sign), float(sigma),
                                  _stream(stream)), "es_qperturb")

    def restore(self, seed, sign, sigma, stream=None):
        _check(load().es_qrestore(self.handle, _u64_arg(seed, "seed"), int(sign), float(sigma),
                                  _stream(stream)), "es_qrestore")

    def swap(self, seed_from, sign_from, seed_to, sign_to, sigma, sigma_to=None, stream=None):
        """Revert member `from` and apply member `to` in one pass: the same
        codes as restore(from) followed by perturb(to)."""
        sigma_to = sigma if sigma_to is None else sigma_to
        _check(load().es_qswap(self.handle, _u64_arg(seed_from, "seed_from"), int(sign_from),
                               float(sigma), _u64_arg(seed_to, "seed_to"), int(sign_to),
                               float(sigma_to), _stream(stream)), "es_qswap")

    def checksum(self, out=None, stream=None):
        """64-bit checksum of the codes (es_qplan_checksum); as Plan.checksum."""
        return _call_checksum(load().es_qplan_checksum, "es_qplan_checksum", self, out, stream)

    def update(self, seeds, signs, rewards, alpha, sigma=0.0, zscore_eps=1e-8, flags=0,
               z_out=None, status_out=None, stream=None, round_seed=0):
        """Update in scale units, always stochastically rounded with the draws
        of round_seed; rewards is a float32 CUDA tensor of len(seeds)."""
        _call_update(load().es_qupdate, "es_qupdate", self.handle, seeds, signs, rewards, alpha,
                     sigma, zscore_eps, flags, z_out, status_out, stream, round_seed)

    def close(self):
        if self._h is not None:
            _check(load().es_qplan_destroy(self._h), "es_qplan_destroy")
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def zscore(rewards, eps=1e-8, out=None, status=None, stream=None):
    """Population z-score of a float32 CUDA tensor (one wavefront, fp64)."""
    out = torch.empty_like(rewards) if out is None else out
    _check(load().es_zscore(_dev_ptr(rewards, torch.float32, "rewards"), rewards.numel(),
                            float(eps), _dev_ptr(out, torch.float32, "out"),
                            _dev_ptr(status, torch.int32, "status"), _stream(stream)), "es_zscore")
    return out


CALIBRATE_READ, CALIBRATE_WRITE, CALIBRATE_READ_WRITE = 0, 1, 2
CALIBRATE_TEMPORAL = 4      # or-ed into a mode: ordinary instead of nontemporal accesses


def hbm_calibrate(buf, mode, sink=None, stream=None):
    """One es_hbm_calibrate pass over the contiguous CUDA tensor `buf` (its
    byte size a multiple of 131072): mode CALIBRATE_READ (the words' XOR is
    folded into `sink`, a one-element int32 CUDA tensor), CALIBRATE_WRITE (buf
    is overwritten) or CALIBRATE_READ_WRITE (buf unchanged), each optionally
    | CALIBRATE_TEMPORAL (ordinary loads and stores instead of nontemporal)."""
    if not buf.is_cuda or not buf.is_contiguous():
        raise ValueError("buf must be a contiguous CUDA tensor")
    sp = None if sink is None else _dev_ptr(sink, torch.int32, "sink")
    _check(load().es_hbm_calibrate(ctypes.c_void_p(buf.data_ptr()),
                                   buf.numel() * buf.element_size(), int(mode), sp,
                                   _stream(stream)), "es_hbm_calibrate")


def sigma_cosine(sigma0, sigma_T, t, T):
    return float(load().es_sigma_cosine(float(sigma0), float(sigma_T), int(t), int(T)))


def philox_words(seed, tensor_id, quad0, n_quads, domain=0, device="cuda", stream=None):
    """Raw Philox words as an int32 CUDA tensor of shape (n_quads, 4)
    (reinterpret as uint32)."""
    out = torch.empty((n_quads, 4), dtype=torch.int32, device=device)
    _check(load().es_philox_words(_u64_arg(seed, "seed"), _u32_arg(tensor_id, "tensor_id"),
                                  _u32_arg(domain, "domain"), _u64_arg(quad0, "quad0"),
                                  _u64_arg(n_quads, "n_quads"), ctypes.c_void_p(out.data_ptr()),
                                  _stream(stream)), "es_philox_words")
    return out


def tile_layout(addr, numel, offset=0):
    """The tiles a plan lays out for one bf16 tensor of `numel` elements at
    device address `addr`, a shard starting `offset` elements into its whole
    tensor (host-side tiling only; nothing is accessed): a list of
    (elem0, end, full, aligned16) in elements of the whole tensor, full
    tiles first."""
    lib = load()
    n = _u64(0)
    off8 = _offset8(offset)
    _check(lib.es_tile_layout(_u64_arg(addr, "addr"), _u64_arg(numel, "numel"), off8, None, 0,
                              ctypes.byref(n)), "es_tile_layout")
    out = (EsTileInfo * max(n.value, 1))()
    _check(lib.es_tile_layout(int(addr), int(numel), off8, out, n.value, ctypes.byref(n)),
           "es_tile_layout")
    return [(t.elem0, t.end, t.full, t.aligned16) for t in out[:n.value]]


def _offset8(offset):
    """A shard's element offset in units of 8 elements (the ABI's offset8)."""
    v = int(offset)
    if v < 0 or v % 8 or v // 8 >= (1 << 32):
        raise ValueError(f"shard offset must be a multiple of 8 in [0, 2^35), got {v}")
    return v // 8


def normals(seed, tensor_id, elem0, n, device="cuda", stream=None):
    """eps_j for j = elem0 .. elem0 + n - 1 of one tensor, float32 CUDA tensor."""
    out = torch.empty(n, dtype=torch.float32, device=device)
    _check(load().es_normals(_u64_arg(seed, "seed"), _u32_arg(tensor_id, "tensor_id"),
                             _u64_arg(elem0, "elem0"), _u64_arg(n, "n"),
                             ctypes.c_void_p(out.data_ptr()), _stream(stream)), "es_normals")
    return out
