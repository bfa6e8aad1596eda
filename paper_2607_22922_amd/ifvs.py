"""Python binding of libifvs (include/ifvs.h): argument marshalling only.

Every step of the search runs in the HIP kernels of libifvs.so; this module
turns torch tensors into device pointers, predicates into the C struct
layout, and status codes into exceptions.  PyTorch provides device memory and
the current HIP stream, nothing else.  There is no fallback: without the
built library (``python -m paper_2607_22922_amd.build``) importing this module
raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libifvs.so")

OK, E_INVALID, E_NOMEM, E_HIP, E_UNSUPPORTED, E_STATE = 0, -1, -2, -3, -4, -5
MEM_HOST, MEM_DEVICE = 0, 1
LUT_F32, LUT_F16 = 0, 1
KSUB = 256
MAX_CLAUSES = 4
MAX_K = 1024
OPT_QTILE, OPT_SPLITS, OPT_PROFILE, OPT_MIN_CHUNK, OPT_GRID_TILES, OPT_GATHER, OPT_GRID_RELATIVE = 1, 2, 3, 4, 5, 6, 7
OPT_SLOT_ORDER = 8
OPT_SHARED_BOUND = 9
OPT_EXACT_PLAN = 10
OPT_SEED_TILES = 11
OPT_COUNT_READS = 12
OPT_COARSE = 13
STAGES = ("condition", "lut", "filter", "scan", "merge", "encode", "coarse")

EXPORTED = ("ifvs_load_index", "ifvs_free_index", "ifvs_select_codebook", "ifvs_build_lut",
            "ifvs_filter", "ifvs_filtered_search", "ifvs_set_option", "ifvs_last_plan",
            "ifvs_read_profile", "ifvs_last_error", "ifvs_load_vectors", "ifvs_exact_search",
            "ifvs_build_sdc_lut", "ifvs_load_reconstructions", "ifvs_train_step", "ifvs_read_params",
            "ifvs_filtered_search_noalloc", "ifvs_read_scan_reads", "ifvs_probe_lds_gather",
            "ifvs_encoder_params", "ifvs_load_encoder", "ifvs_encode_predicates",
            "ifvs_build_coarse", "ifvs_lut_bounds", "ifvs_filtered_search_bounded", "ifvs_read_coarse",
            "ifvs_last_coarse", "ifvs_query_batch")


class IfvsError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"ifvs status {status}: {message}")
        self.status = status


class IndexDesc(ctypes.Structure):
    _fields_ = [
        ("n", ctypes.c_int64),
        ("dim", ctypes.c_int32),
        ("m", ctypes.c_int32),
        ("ksub", ctypes.c_int32),
        ("n_attr", ctypes.c_int32),
        ("codes", ctypes.c_void_p),
        ("codebook", ctypes.c_void_p),
        ("attrs", ctypes.c_void_p),
        ("bank_rows", ctypes.c_int32),
        ("r", ctypes.c_int32),
        ("h", ctypes.c_int32),
        ("mem_kind", ctypes.c_int32),
        ("hash_seed", ctypes.c_uint64),
        ("bank", ctypes.c_void_p),
        ("W", ctypes.c_void_p),
        ("max_batch", ctypes.c_int32),
        ("max_k", ctypes.c_int32),
        ("n_cluster", ctypes.c_int32),
        ("cluster_col", ctypes.c_int32 * 2),
    ]


class Clause(ctypes.Structure):
    _fields_ = [("col", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("lo", ctypes.c_int64), ("hi", ctypes.c_int64)]


class Predicate(ctypes.Structure):
    _fields_ = [("n_clauses", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("c", Clause * MAX_CLAUSES)]


class EncoderDesc(ctypes.Structure):
    _fields_ = [
        ("hidden", ctypes.c_int32),
        ("heads", ctypes.c_int32),
        ("layers", ctypes.c_int32),
        ("ffn", ctypes.c_int32),
        ("n_params", ctypes.c_int64),
        ("params", ctypes.c_void_p),
        ("col_offset", ctypes.c_void_p),
        ("col_scale", ctypes.c_void_p),
        ("mem_kind", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
    ]


def _load_library() -> ctypes.CDLL:
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is missing: build it with "
                          "`python -m paper_2607_22922_amd.build` (there is no fallback path)")
    lib = ctypes.CDLL(_LIB_PATH)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    sig = {
        "ifvs_load_index": ([ctypes.POINTER(IndexDesc), ctypes.POINTER(vp)], i32),
        "ifvs_free_index": ([vp], None),
        "ifvs_select_codebook": ([vp, i32, vp, vp, vp, vp, vp, vp], i32),
        "ifvs_build_lut": ([vp, i32, vp, vp, vp, i32, vp, vp], i32),
        "ifvs_filter": ([vp, i32, vp, vp, vp, vp], i32),
        "ifvs_filtered_search": ([vp, i32, vp, vp, i32, i32, vp, vp, vp, vp], i32),
        "ifvs_filtered_search_noalloc": ([vp, i32, vp, vp, i32, i32, vp, vp, vp, vp], i32),
        "ifvs_set_option": ([vp, i32, i64], i32),
        "ifvs_last_plan": ([vp, ctypes.POINTER(ctypes.c_int64)], i32),
        "ifvs_read_profile": ([vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)], i32),
        "ifvs_last_error": ([], ctypes.c_char_p),
        "ifvs_load_vectors": ([vp, vp, i32], i32),
        "ifvs_build_sdc_lut": ([vp, i32, vp, i32, vp, vp], i32),
        "ifvs_load_reconstructions": ([vp], i32),
        "ifvs_exact_search": ([vp, i32, vp, vp, i32, vp, vp, vp], i32),
        "ifvs_train_step": ([vp, i32, vp, vp, vp, vp, i32, i32, ctypes.c_float, ctypes.c_float, ctypes.c_float,
                             vp, vp, vp], i32),
        "ifvs_read_params": ([vp, vp, vp, vp], i32),
        "ifvs_read_scan_reads": ([vp, ctypes.POINTER(ctypes.c_int64), vp], i32),
        "ifvs_probe_lds_gather": ([i32, ctypes.POINTER(ctypes.c_double), vp], i32),
        "ifvs_encoder_params": ([i32, i32, i32, i32, i32, i32], i64),
        "ifvs_load_encoder": ([vp, ctypes.POINTER(EncoderDesc)], i32),
        "ifvs_encode_predicates": ([vp, i32, vp, vp, vp], i32),
        "ifvs_build_coarse": ([vp, i32, i32], i32),
        "ifvs_lut_bounds": ([vp, i32, vp, vp, vp, vp], i32),
        "ifvs_filtered_search_bounded": ([vp, i32, vp, vp, i32, vp, vp, i32, vp, vp, vp, vp], i32),
        "ifvs_query_batch": ([vp, i32, vp, vp, vp, vp, vp, vp, i32, vp, i32, vp, vp, vp], i32),
        "ifvs_read_coarse": ([vp, ctypes.POINTER(i32), vp, vp, vp], i32),
        "ifvs_last_coarse": ([vp, ctypes.POINTER(i32)], i32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


_lib = _load_library()


def lib() -> ctypes.CDLL:
    return _lib


def _check(status: int) -> None:
    if status != OK:
        raise IfvsError(status, _lib.ifvs_last_error().decode(errors="replace"))


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def probe_lds_gather(active_lanes: int, stream=None) -> float:
    """ifvs_probe_lds_gather: chip-wide wavefront reads per second of random
    4-byte LDS reads with `active_lanes` lanes each (a GPU measurement)."""
    out = ctypes.c_double()
    _check(_lib.ifvs_probe_lds_gather(int(active_lanes), ctypes.byref(out), _stream(stream)))
    return out.value


def pack_predicates(preds) -> ctypes.Array:
    """List of clause lists [(col, lo, hi), ...] -> C array of ifvs_predicate."""
    arr = (Predicate * max(1, len(preds)))()
    for i, clauses in enumerate(preds):
        if len(clauses) > MAX_CLAUSES:
            arr[i].n_clauses = len(clauses)      # rejected by the library
            continue
        arr[i].n_clauses = len(clauses)
        for j, (col, lo, hi) in enumerate(clauses):
            arr[i].c[j].col = int(col)
            arr[i].c[j].lo = int(lo)
            arr[i].c[j].hi = int(hi)
    return arr


def _dev_f32(t, device):
    return t.to(device=device, dtype=torch.float32).contiguous()


class Index:
    """A PQ-quantized dataset resident on one GPU (ifvs_load_index)."""

    def __init__(self, codes, C_pq, attrs=None, bank=None, W=None, r=0, h=0, hash_seed=0,
                 max_batch=256, max_k=100, cluster_cols=()):
        codes = codes.contiguous()
        device = codes.device
        self.mem_kind = MEM_DEVICE if device.type == "cuda" else MEM_HOST
        n, m = codes.shape
        M, ksub, dsub = C_pq.shape
        assert M == m and ksub == KSUB, "C_pq must be [m][256][dsub]"
        self._keep = []                                  # host/device arrays alive during load
        cb = C_pq.to(device=device, dtype=torch.float32).contiguous()
        at = None if attrs is None else attrs.to(device=device, dtype=torch.int32).contiguous()
        bk = None if bank is None else bank.to(device=device, dtype=torch.float32).contiguous()
        Wt = None if W is None else W.to(device=device, dtype=torch.float32).contiguous()
        self._keep += [codes, cb, at, bk, Wt]
        d = IndexDesc()
        d.n, d.dim, d.m, d.ksub = n, m * dsub, m, KSUB
        d.n_attr = 0 if at is None else at.shape[0]
        d.codes, d.codebook, d.attrs = codes.data_ptr(), cb.data_ptr(), _ptr(at)
        d.bank_rows = 0 if bk is None else bk.shape[0]
        d.r, d.h, d.hash_seed = (int(r), int(h), int(hash_seed)) if bk is not None else (0, 0, 0)
        d.mem_kind = self.mem_kind
        d.bank, d.W = _ptr(bk), _ptr(Wt)
        d.max_batch, d.max_k = int(max_batch), int(max_k)
        d.n_cluster = len(cluster_cols)
        for i, c in enumerate(cluster_cols):
            d.cluster_col[i] = int(c)
        handle = ctypes.c_void_p()
        _check(_lib.ifvs_load_index(ctypes.byref(d), ctypes.byref(handle)))
        self._keep = None
        self.handle = handle
        self.n, self.m, self.dsub, self.dim = n, m, dsub, m * dsub
        self.n_attr = d.n_attr
        self.bank_rows, self.r = d.bank_rows, d.r
        self.max_batch, self.max_k = int(max_batch), int(max_k)
        self.device = torch.device("cuda", torch.cuda.current_device())

    @classmethod
    def from_workload(cls, w, max_batch=256, max_k=None, conditioned=True, cluster_cols=()):
        return cls(w.codes, w.C_pq, w.attrs, w.bank if conditioned else None,
                   w.W if conditioned else None, w.r, w.h, w.hash_seed,
                   max_batch=max_batch, max_k=max_k or w.k, cluster_cols=cluster_cols)

    def close(self):
        if getattr(self, "handle", None) is not None and self.handle.value:
            _lib.ifvs_free_index(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---------------------------------------------------------- raw calls
    def set_option(self, option: int, value: int) -> None:
        _check(_lib.ifvs_set_option(self.handle, option, int(value)))

    def last_plan(self) -> dict:
        """Launch plan of the most recent filtered_search on this index."""
        out = (ctypes.c_int64 * 5)()
        _check(_lib.ifvs_last_plan(self.handle, out))
        return dict(qtile=out[0], splits=out[1], min_chunk=out[2], lds_bytes=out[3], grid_tiles=out[4])

    def last_coarse(self) -> bool:
        """Whether the most recent filtered search ran the coarse bound."""
        out = ctypes.c_int32()
        _check(_lib.ifvs_last_coarse(self.handle, ctypes.byref(out)))
        return bool(out.value)

    def build_coarse(self, n_centroids: int, iters: int = 20) -> None:
        """ifvs_build_coarse: the coarse quantizer of the exact pruning bound."""
        _check(_lib.ifvs_build_coarse(self.handle, int(n_centroids), int(iters)))

    def read_coarse(self):
        """(assign [n] int32, radius [n] fp32, centroid codes [C][m] uint8),
        host numpy arrays by vector id (ifvs_read_coarse)."""
        c = ctypes.c_int32()
        _check(_lib.ifvs_read_coarse(self.handle, ctypes.byref(c), None, None, None))
        assign = np.empty(self.n, dtype=np.int32)
        radius = np.empty(self.n, dtype=np.float32)
        codes = np.empty((c.value, self.m), dtype=np.uint8)
        _check(_lib.ifvs_read_coarse(self.handle, None, assign.ctypes.data, radius.ctypes.data,
                                     codes.ctypes.data))
        return assign, radius, codes

    def lut_bounds_into(self, nq, alpha, wf, bounds_out, stream=None):
        _check(_lib.ifvs_lut_bounds(self.handle, nq, _ptr(alpha), _ptr(wf), bounds_out.data_ptr(),
                                    _stream(stream)))

    def lut_bounds(self, nq, alpha=None, wf=None):
        """[nq][2] factors of the coarse bound for tables built with alpha, wf."""
        out = torch.empty(nq, 2, device=self.device, dtype=torch.float32)
        self.lut_bounds_into(nq, alpha, wf, out)
        return out

    def search_bounded_into(self, nq, preds_c, lut, lut_dtype, alpha, wf, k, ids_out, dist_out, bitmap_out=None,
                            stream=None):
        """ifvs_filtered_search_bounded: alpha and wf are the operands the
        tables were built with (None for none)."""
        _check(_lib.ifvs_filtered_search_bounded(self.handle, nq, preds_c, lut.data_ptr(), lut_dtype,
                                                 _ptr(alpha), _ptr(wf), k, ids_out.data_ptr(), dist_out.data_ptr(),
                                                 _ptr(bitmap_out), _stream(stream)))

    def search_bounded(self, preds, lut, alpha, wf, k, lut_dtype=LUT_F32):
        nq = len(preds)
        ids = torch.empty(nq, k, device=self.device, dtype=torch.int32)
        dist = torch.empty(nq, k, device=self.device, dtype=torch.float32)
        self.search_bounded_into(nq, pack_predicates(preds), lut, lut_dtype, alpha, wf, k, ids, dist)
        return ids, dist

    def query_batch_into(self, q, preds_c, w_z, wz_out, alpha_out, wf_out, lut_dtype, lut_out, k, ids_out,
                         dist_out, stream=None):
        """ifvs_query_batch: encoder (when w_z is None), condition, tables
        and the bounded search in one call."""
        _check(_lib.ifvs_query_batch(self.handle, q.shape[0], q.data_ptr(), preds_c, _ptr(w_z), _ptr(wz_out),
                                     _ptr(alpha_out), wf_out.data_ptr(), lut_dtype, lut_out.data_ptr(), k,
                                     ids_out.data_ptr(), dist_out.data_ptr(), _stream(stream)))

    def read_profile(self) -> dict:
        """Per-stage (total kernel ms, launches) since the last read."""
        ms = (ctypes.c_double * len(STAGES))()
        n = (ctypes.c_int64 * len(STAGES))()
        _check(_lib.ifvs_read_profile(self.handle, ms, n))
        return {name: (ms[i], n[i]) for i, name in enumerate(STAGES)}

    def load_encoder(self, enc: dict) -> None:
        """ifvs_load_encoder from a dict of weights (the names of the layout
        in ifvs.h; per-layer weights under "layers", a list of dicts with
        Wq, Wk, Wv, bq, bk, bv, Wo, bo, ln1_g, ln1_b, ln2_g, ln2_b, W1, b1,
        W2, b2).  Packs them in the documented order (host memory)."""
        H, F = int(enc["cls"].shape[0]), int(enc["layers"][0]["W1"].shape[1])
        heads, layers = int(enc["heads"]), len(enc["layers"])
        f = lambda t: torch.as_tensor(t).detach().to("cpu", torch.float32).reshape(-1)
        parts = [f(enc["col_embed"]), f(enc["feat_w"]), f(enc["feat_b"]), f(enc["cls"])]
        for p in enc["layers"]:
            wqkv = torch.cat([torch.as_tensor(p[k]).detach().cpu().float() for k in ("Wq", "Wk", "Wv")], dim=1)
            bqkv = torch.cat([torch.as_tensor(p[k]).detach().cpu().float() for k in ("bq", "bk", "bv")])
            parts += [f(p["ln1_g"]), f(p["ln1_b"]), f(wqkv), f(bqkv), f(p["Wo"]), f(p["bo"]),
                      f(p["ln2_g"]), f(p["ln2_b"]), f(p["W1"]), f(p["b1"]), f(p["W2"]), f(p["b2"])]
        parts += [f(enc["lnf_g"]), f(enc["lnf_b"]), f(enc["out_w"]), f(enc["out_b"])]
        packed = torch.cat(parts).contiguous()
        off = torch.as_tensor(enc["col_offset"]).detach().to("cpu", torch.float64).contiguous()
        sc = torch.as_tensor(enc["col_scale"]).detach().to("cpu", torch.float64).contiguous()
        d = EncoderDesc()
        d.hidden, d.heads, d.layers, d.ffn = H, heads, layers, F
        d.n_params = packed.numel()
        d.params, d.col_offset, d.col_scale = packed.data_ptr(), off.data_ptr(), sc.data_ptr()
        d.mem_kind = MEM_HOST
        _check(_lib.ifvs_load_encoder(self.handle, ctypes.byref(d)))

    def encode_predicates_into(self, nq, preds_c, wz_out, stream=None):
        _check(_lib.ifvs_encode_predicates(self.handle, nq, preds_c, wz_out.data_ptr(), _stream(stream)))

    def encode_predicates(self, preds):
        """w_z [nq][dim] of each predicate through the attached encoder."""
        wz = torch.empty(len(preds), self.dim, device=self.device, dtype=torch.float32)
        self.encode_predicates_into(len(preds), pack_predicates(preds), wz)
        return wz

    def read_scan_reads(self, stream=None) -> list:
        """With OPT_COUNT_READS on: [66] table reads issued with n active
        lanes (index n), tiles summed ([0]) and tiles the list scan read
        whole ([65]) since the last read."""
        out = (ctypes.c_int64 * 66)()
        _check(_lib.ifvs_read_scan_reads(self.handle, out, _stream(stream)))
        return list(out)

    def select_codebook_into(self, q, preds_c, w_z, alpha_out, wf_out, stream=None):
        _check(_lib.ifvs_select_codebook(self.handle, q.shape[0], q.data_ptr(), preds_c,
                                         _ptr(w_z), _ptr(alpha_out), wf_out.data_ptr(),
                                         _stream(stream)))

    def build_lut_into(self, q, alpha, wf, lut_dtype, lut_out, stream=None):
        _check(_lib.ifvs_build_lut(self.handle, q.shape[0], q.data_ptr(), _ptr(alpha), _ptr(wf),
                                   lut_dtype, lut_out.data_ptr(), _stream(stream)))

    def build_sdc_lut_into(self, q, lut_dtype, lut_out, stream=None):
        _check(_lib.ifvs_build_sdc_lut(self.handle, q.shape[0], q.data_ptr(), lut_dtype, lut_out.data_ptr(),
                                       _stream(stream)))

    def filter_into(self, nq, preds_c, bitmap_out, count_out=None, stream=None):
        _check(_lib.ifvs_filter(self.handle, nq, preds_c, bitmap_out.data_ptr(), _ptr(count_out),
                                _stream(stream)))

    def search_into(self, nq, preds_c, lut, lut_dtype, k, ids_out, dist_out, bitmap_out=None,
                    stream=None):
        _check(_lib.ifvs_filtered_search(self.handle, nq, preds_c, lut.data_ptr(), lut_dtype, k,
                                         ids_out.data_ptr(), dist_out.data_ptr(), _ptr(bitmap_out),
                                         _stream(stream)))

    def search_noalloc_into(self, nq, preds_c, lut, lut_dtype, k, ids_out, dist_out, bitmap_out=None,
                            stream=None):
        """ifvs_filtered_search_noalloc: the same search with the library's
        static workspace (no allocation in the call)."""
        _check(_lib.ifvs_filtered_search_noalloc(self.handle, nq, preds_c, lut.data_ptr(), lut_dtype, k,
                                                 ids_out.data_ptr(), dist_out.data_ptr(), _ptr(bitmap_out),
                                                 _stream(stream)))

    def load_vectors(self, x):
        """Attach the full-precision vectors [n][dim] (ifvs_load_vectors)."""
        x = x.to(dtype=torch.float32).contiguous()
        _check(_lib.ifvs_load_vectors(self.handle, x.data_ptr(),
                                      MEM_DEVICE if x.device.type == "cuda" else MEM_HOST))

    def train_step_into(self, q, preds_c, w_z, cand, n_pos, tau, lam, lr, loss_out, dwz_out=None, stream=None):
        """One SGD step of the memory bank and W (ifvs_train_step)."""
        _check(_lib.ifvs_train_step(self.handle, q.shape[0], q.data_ptr(), preds_c, _ptr(w_z), cand.data_ptr(),
                                    cand.shape[1], int(n_pos), float(tau), float(lam), float(lr),
                                    loss_out.data_ptr(), _ptr(dwz_out), _stream(stream)))

    def train_step(self, q, preds, w_z, cand, n_pos, tau, lam, lr, want_dwz=False):
        """Marshalling wrapper: returns (per-query loss, dL/dw_z or None)."""
        q = q.contiguous()
        cand = cand.to(dtype=torch.int32).contiguous()
        loss = torch.empty(q.shape[0], device=self.device)
        dwz = torch.empty_like(q) if want_dwz else None
        self.train_step_into(q, pack_predicates(preds), None if w_z is None else w_z.contiguous(), cand, n_pos,
                             tau, lam, lr, loss, dwz)
        return loss, dwz

    def read_params(self):
        """The current memory bank [bank_rows][m*r] and W [m][r][256][dsub] (ifvs_read_params)."""
        bank = torch.empty(self.bank_rows, self.m * self.r, device=self.device)
        W = torch.empty(self.m, self.r, 256, self.dsub, device=self.device)
        _check(_lib.ifvs_read_params(self.handle, bank.data_ptr(), W.data_ptr(), _stream(None)))
        return bank, W

    def load_reconstructions(self):
        """Attach the reconstructions of the codes (ifvs_load_reconstructions)."""
        _check(_lib.ifvs_load_reconstructions(self.handle))

    def exact_search_into(self, q, preds_c, k, ids_out, dist_out, stream=None):
        _check(_lib.ifvs_exact_search(self.handle, q.shape[0], q.data_ptr(), preds_c, k,
                                      ids_out.data_ptr(), dist_out.data_ptr(), _stream(stream)))

    # ------------------------------------------------ allocating helpers
    def words(self) -> int:
        return (self.n + 31) // 32

    def select_codebook(self, q, preds, w_z=None):
        nq = q.shape[0]
        q = _dev_f32(q, self.device)
        w_z = None if w_z is None else _dev_f32(w_z, self.device)
        alpha = (torch.empty(nq, self.m * self.r, device=self.device)
                 if self.bank_rows > 0 else None)
        wf = torch.empty(nq, self.dim, device=self.device)
        self.select_codebook_into(q, pack_predicates(preds), w_z, alpha, wf)
        return alpha, wf

    def query_batch(self, q, preds, k, w_z=None, lut_dtype=LUT_F32):
        """Returns (ids, dist, w_z, alpha, w_f, lut); w_z is the encoder's
        output when none is given, else the argument."""
        nq = q.shape[0]
        q = _dev_f32(q, self.device)
        wz = torch.empty(nq, self.dim, device=self.device) if w_z is None else _dev_f32(w_z, self.device)
        alpha = (torch.empty(nq, self.m * self.r, device=self.device)
                 if self.bank_rows > 0 else None)
        wf = torch.empty(nq, self.dim, device=self.device)
        dt = torch.float16 if lut_dtype == LUT_F16 else torch.float32
        lut = torch.empty(nq, self.m, KSUB, device=self.device, dtype=dt)
        ids = torch.empty(nq, k, device=self.device, dtype=torch.int32)
        dist = torch.empty(nq, k, device=self.device, dtype=torch.float32)
        self.query_batch_into(q, pack_predicates(preds), None if w_z is None else wz,
                              wz if w_z is None else None, alpha, wf, lut_dtype, lut, k, ids, dist)
        return ids, dist, wz, alpha, wf, lut

    def build_lut(self, q, alpha=None, wf=None, lut_dtype=LUT_F32):
        nq = q.shape[0]
        q = _dev_f32(q, self.device)
        dt = torch.float16 if lut_dtype == LUT_F16 else torch.float32
        lut = torch.empty(nq, self.m, KSUB, device=self.device, dtype=dt)
        self.build_lut_into(q, alpha, wf, lut_dtype, lut)
        return lut

    def build_sdc_lut(self, q, lut_dtype=LUT_F32):
        """Symmetric distance tables (query quantized with the codebook)."""
        nq = q.shape[0]
        q = _dev_f32(q, self.device)
        dt = torch.float16 if lut_dtype == LUT_F16 else torch.float32
        lut = torch.empty(nq, self.m, KSUB, device=self.device, dtype=dt)
        self.build_sdc_lut_into(q, lut_dtype, lut)
        return lut

    def filter(self, preds):
        nq = len(preds)
        bm = torch.empty(nq, self.words(), device=self.device, dtype=torch.int32)
        cnt = torch.empty(nq, device=self.device, dtype=torch.int64)
        self.filter_into(nq, pack_predicates(preds), bm, cnt)
        return bm, cnt

    def search(self, preds, lut, k, lut_dtype=LUT_F32, want_bitmap=False):
        nq = len(preds)
        ids = torch.empty(nq, k, device=self.device, dtype=torch.int32)
        dist = torch.empty(nq, k, device=self.device, dtype=torch.float32)
        bm = (torch.empty(nq, self.words(), device=self.device, dtype=torch.int32)
              if want_bitmap else None)
        self.search_into(nq, pack_predicates(preds), lut, lut_dtype, k, ids, dist, bm)
        return (ids, dist, bm) if want_bitmap else (ids, dist)

    def exact_search(self, q, preds, k):
        """Exact filtered kNN over the attached full-precision vectors."""
        nq = len(preds)
        q = _dev_f32(q, self.device)
        ids = torch.empty(nq, k, device=self.device, dtype=torch.int32)
        dist = torch.empty(nq, k, device=self.device, dtype=torch.float32)
        self.exact_search_into(q, pack_predicates(preds), k, ids, dist)
        return ids, dist

    def query(self, q, preds, k, w_z=None, lut_dtype=LUT_F32, conditioned=True):
        """All four steps for one batch: condition, table, filter+scan+select."""
        alpha, wf = self.select_codebook(q, preds, w_z)
        lut = self.build_lut(q, alpha if conditioned else None, wf, lut_dtype)
        return self.search(preds, lut, k, lut_dtype)


def bitmap_words_to_numpy(bm: torch.Tensor) -> np.ndarray:
    """Device int32 words -> host uint32 words (same bits)."""
    return bm.cpu().numpy().view(np.uint32)
