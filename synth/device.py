"""Binding of the device input generator and copy kernel (synth/synth.hip)."""
from __future__ import annotations

import ctypes
import os

import torch  # before libsynth.so: share PyTorch's HIP runtime

from . import gen

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsynth.so")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run "
                          "`python -m paper_2607_21224_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i, i64, u64, u32, f = (ctypes.c_void_p, ctypes.c_int, ctypes.c_int64,
                               ctypes.c_uint64, ctypes.c_uint32, ctypes.c_float)
    lib.synth_fill_normal.argtypes = [vp, i, i64, i64, u64, i, i64, f, u32, f, vp]
    lib.synth_fill_normal.restype = i
    lib.synth_copy_f32.argtypes = [vp, vp, i64, vp]
    lib.synth_copy_f32.restype = i
    lib.synth_shape_stream.argtypes = [vp, i, i, i64, i64, i64, i, i, i, u32, vp, vp]
    lib.synth_shape_stream.restype = i
    lib.synth_shape_sync.argtypes = [vp, i, i, i, i, i, i, i64, u32, vp, vp]
    lib.synth_shape_sync.restype = i
    return lib


_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = _load()
    return _lib


def _check_f32_device(x, name: str) -> None:
    """The kernels write through the raw address: only a contiguous fp32
    tensor on the GPU may reach them."""
    if x.dtype != torch.float32 or not x.is_contiguous() or not x.is_cuda:
        raise ValueError(f"{name} must be a contiguous float32 GPU tensor")


def _stream(s):
    if s is None:
        return None
    return s if isinstance(s, int) else int(s.cuda_stream)


def fill_normal(out, P: int, seed: int, kind: int, t: int, sigma: float,
                outlier_rate: float = 0.0, outlier_scale: float = 100.0,
                stream=None) -> None:
    """Fill out[:, :P] (a contiguous (rows, ld) fp32 CUDA tensor) with stream
    key(seed, kind, t, row) draws."""
    _check_f32_device(out, "out")
    if out.dim() not in (1, 2):
        raise ValueError("out must be a (ld,) or (rows, ld) tensor")
    rows, ld = (out.shape[0], out.shape[1]) if out.dim() == 2 else (1, out.shape[0])
    if not 0 <= P <= ld:
        raise ValueError(f"P = {P} does not fit rows of {ld}")
    r = lib().synth_fill_normal(out.data_ptr(), rows, P, ld, seed, kind, t, sigma,
                                gen.outlier_threshold(outlier_rate), outlier_scale,
                                _stream(stream))
    if r != 0:
        raise RuntimeError(f"synth_fill_normal failed ({r})")


def fill_theta0(out, P: int, seed: int, sigma: float = 0.02, stream=None) -> None:
    fill_normal(out, P, seed, gen.KIND_THETA0, 0, sigma, stream=stream)


def fill_grads(out, P: int, seed: int, step: int, sigma: float = 1e-3,
               outlier_rate: float = 0.0, outlier_scale: float = 100.0,
               stream=None) -> None:
    fill_normal(out, P, seed, gen.KIND_GRAD, step, sigma, outlier_rate,
                outlier_scale, stream)


def copy_f32(dst, src, n: int, stream=None) -> None:
    _check_f32_device(dst, "dst")
    _check_f32_device(src, "src")
    if not 0 <= n <= min(dst.numel(), src.numel()):
        raise ValueError(f"copy of {n} elements between tensors of {src.numel()} and "
                         f"{dst.numel()}")
    r = lib().synth_copy_f32(dst.data_ptr(), src.data_ptr(), n, _stream(stream))
    if r != 0:
        raise RuntimeError(f"synth_copy_f32 failed ({r})")


# ---- traffic-shape kernel -----------------------------------------------------

SHAPE_MAX_READ = 256
SHAPE_MAX_WRITE_ONLY = 64


class ShapeRow:
    """One row of a traffic shape: coordinates [0, P) of ``tensor`` starting
    at element ``offset`` (plain rows), or the row's segment in every tile of
    a tile-major layout.  ``write`` = the row is written back in place after
    it is read; ``read`` = False makes a write-only row (fp32)."""

    def __init__(self, tensor, offset: int = 0, write: bool = False, read: bool = True):
        if not isinstance(tensor, torch.Tensor) or not tensor.is_cuda or not tensor.is_contiguous():
            raise ValueError("a shape row lives in a contiguous GPU tensor")
        if tensor.dtype not in (torch.float32, torch.bfloat16):
            raise ValueError("shape rows are float32 or bfloat16")
        if not read and (write or tensor.dtype != torch.float32):
            raise ValueError("a write-only row is a float32 row")
        self.tensor, self.offset, self.write, self.read = tensor, int(offset), bool(write), bool(read)

    @property
    def esize(self) -> int:
        return self.tensor.element_size()

    def nbytes(self, P: int) -> int:
        """Bytes the pass moves on this row."""
        return P * self.esize * (int(self.read) + int(self.write or not self.read))


class ShapePass:
    """A traffic shape ready to launch: the device row table and the checks
    that every row covers what the kernel touches."""

    def __init__(self, rows, P: int, tile: int = 0, tile_stride: int = 0,
                 xcd: bool = False, batch: int = 8, threads: int = 64):
        rows = list(rows)
        rd = [r for r in rows if r.read]
        wo = [r for r in rows if not r.read]
        if not 1 <= len(rows) or len(rd) > SHAPE_MAX_READ or len(wo) > SHAPE_MAX_WRITE_ONLY:
            raise ValueError(f"{len(rd)} read and {len(wo)} write-only rows: at most "
                             f"{SHAPE_MAX_READ} and {SHAPE_MAX_WRITE_ONLY}")
        if P < 0 or P % 4:
            raise ValueError(f"P = {P} must be a non-negative multiple of 4")
        if batch not in (8, 16):
            raise ValueError("batch is 8 or 16")
        if threads not in (64, 128, 256, 512, 1024):
            raise ValueError("threads per block is a power of two in [64, 1024]")
        if tile and (tile % (4 * threads) or tile_stride < 0):
            raise ValueError("tile is a multiple of 4 * threads coordinates")
        dev = rows[0].tensor.device
        t = tile if tile else max(P, 1)
        for r in rows:
            if r.tensor.device != dev:
                raise ValueError("all rows on one device")
            if tile and tile_stride % r.esize:
                raise ValueError("tile_stride is a whole number of elements")
            ts = tile_stride // r.esize if tile else 0
            if P:
                last = r.offset + ((P - 1) // t) * ts + (P - 1) % t
                if r.offset < 0 or last >= r.tensor.numel():
                    raise ValueError(f"row at element {r.offset} reaches element {last} of a "
                                     f"tensor of {r.tensor.numel()}")
            # 16-byte (fp32) / 8-byte (bf16) vector accesses at every 4th coordinate
            if (r.tensor.data_ptr() + r.offset * r.esize) % (4 * r.esize):
                raise ValueError("row start not aligned for 4-coordinate vectors")
            if tile and tile_stride % (4 * r.esize):
                raise ValueError("tile_stride not aligned for 4-coordinate vectors")
        words = []
        for r in rd:
            a = r.tensor.data_ptr() + r.offset * r.esize
            words += [a, a if r.write else 0, 1 if r.esize == 2 else 0]
        words += [r.tensor.data_ptr() + r.offset * r.esize for r in wo]
        self.table = torch.tensor(words, dtype=torch.int64, device=dev)
        self.sink = torch.zeros(256, dtype=torch.int32, device=dev)
        self.keep_rows = rows  # the rows (and their tensors) outlive the pass
        self.n_rd, self.n_wo = len(rd), len(wo)
        self.P, self.tile, self.tile_stride = P, tile, tile_stride
        self.xcd, self.batch, self.threads = int(bool(xcd)), batch, threads
        self.bytes = sum(r.nbytes(P) for r in rows)

    def launch(self, stream=None, sentinel: int = 0x9E3779B9) -> None:
        r = lib().synth_shape_stream(self.table.data_ptr(), self.n_rd, self.n_wo, self.P,
                                     self.tile, self.tile_stride, self.xcd, self.batch,
                                     self.threads, sentinel, self.sink.data_ptr(),
                                     _stream(stream))
        if r != 0:
            raise RuntimeError(f"synth_shape_stream failed ({r})")


SYNC_KINDS = {"cpdp": 0, "localsgd": 1, "ddp": 2}
SYNC_ORDER_W = (4, 8, 16, 32)


class ShapeSyncPass(ShapePass):
    """The rows of a synchronisation step (as bench.sync_shape_rows lists
    them) streamed in the library's own load and store order with no
    arithmetic (shape_sync_kernel in synth/synth.hip).  The rows must follow
    the kernel's fixed pattern for ``method`` with W replicas; anything else
    is refused before a launch."""

    def __init__(self, rows, P: int, method: str, adamw: bool, W: int):
        rows = list(rows)
        super().__init__(rows, P)
        if method not in SYNC_KINDS:
            raise ValueError(f"method {method!r}: one of {sorted(SYNC_KINDS)}")
        if W not in SYNC_ORDER_W:
            raise ValueError(f"W = {W}: the order kernel is built for W in {SYNC_ORDER_W}")
        if P * 4 >= 2 ** 32:
            raise ValueError(f"P = {P}: byte offsets must fit 32 bits")
        R = 3 if adamw else 2
        fam = ["m", "v", "t"] if adamw else ["m", "t"]
        if method == "localsgd":
            roles = [r for _ in range(W) for r in ["g"] + fam]
        else:
            roles = ["g"] * W + fam * W + (["u", "a"] if method == "cpdp" else [])
        rd = [r for r in rows if r.read]
        wo = [r for r in rows if not r.read]
        if len(rd) != len(roles) or len(wo) != (1 if method == "localsgd" else 0):
            raise ValueError(f"{len(rd)} read and {len(wo)} write-only rows do not follow the "
                             f"{method} pattern at W = {W} ({len(roles)} read rows)")
        narrow = {}
        for role, r in zip(roles, rd):
            if r.write != (role != "g"):
                raise ValueError(f"row {role}: written back = {r.write}, the pattern says "
                                 f"{role != 'g'}")
            n = r.esize == 2
            if narrow.setdefault(role, n) != n:
                raise ValueError(f"the {role} rows mix bf16 and fp32")
        if narrow.get("v", False) or narrow.get("u", False) or narrow.get("a", False):
            raise ValueError("second-moment, SlowMo and anchor rows are fp32")
        if (narrow["g"] or narrow["m"]) and (method != "cpdp" or adamw):
            raise ValueError("bf16 gradient or momentum rows only on the momentum-SGD reconcile")
        self.kind, self.adam, self.W, self.R = SYNC_KINDS[method], int(bool(adamw)), W, R
        self.np, self.ng, self.nm = int(narrow["t"]), int(narrow["g"]), int(narrow["m"])

    def launch(self, stream=None, sentinel: int = 0x9E3779B9) -> None:
        r = lib().synth_shape_sync(self.table.data_ptr(), self.kind, self.adam, self.W, self.np,
                                   self.ng, self.nm, self.P, sentinel, self.sink.data_ptr(),
                                   _stream(stream))
        if r != 0:
            raise RuntimeError(f"synth_shape_sync failed ({r})")
