"""Thin ctypes binding of libtcl (include/tcl.h): argument marshalling only.

Every step of the cost model runs in libtcl's HIP kernels; this module only
converts torch tensors to device pointers and the caller's current HIP
stream, and raises on a non-OK status. Loading fails loudly if the library
has not been built: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtcl.so")
_lib = None

TCL_F32, TCL_BF16 = 0, 1
TCL_F32_MATMUL_SPLIT, TCL_F32_MATMUL_NATIVE, TCL_F32_MATMUL_SPLIT_BF16 = 0, 1, 2
F32_MATMUL = {"split": TCL_F32_MATMUL_SPLIT, "native": TCL_F32_MATMUL_NATIVE,
              "split_bf16": TCL_F32_MATMUL_SPLIT_BF16}
STATUS = {0: "TCL_OK", -1: "TCL_ERR_INVALID_ARG", -2: "TCL_ERR_UNSUPPORTED", -3: "TCL_ERR_WORKSPACE",
          -4: "TCL_ERR_OOM", -5: "TCL_ERR_HIP"}


class TclError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class Config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("F", "d_model", "d_inner", "d_state", "d_conv", "dt_rank", "n_layers", "head_hidden",
                 "final_norm")] + [("norm_eps", ctypes.c_float), ("dtype", ctypes.c_int32),
                                   ("f32_matmul", ctypes.c_int32), ("enc_hidden", ctypes.c_int32 * 2),
                                   ("dec_hidden2", ctypes.c_int32)]


class KDLoss(ctypes.Structure):
    """tcl_kd_loss: the Eq. (9) distillation objective."""
    _fields_ = [("beta", ctypes.c_float), ("phi", ctypes.c_float), ("sigma", ctypes.c_float),
                ("ewc_lambda", ctypes.c_float), ("d_fisher", ctypes.c_void_p), ("d_theta_prev", ctypes.c_void_p),
                ("d_phi", ctypes.c_void_p)]


_vp, _i32, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
_SIGS = {
    "tcl_param_count": (_sz, [ctypes.POINTER(Config)]),
    "tcl_cost_model_create": (_i32, [ctypes.POINTER(Config), _vp, _sz, ctypes.POINTER(_vp)]),
    "tcl_cost_model_destroy": (_i32, [_vp]),
    "tcl_score_workspace_bytes": (_sz, [_vp, _i32, _i32]),
    "tcl_set_score_streams": (_i32, [_vp, _i32]),
    "tcl_score": (_i32, [_vp, _i32, _i32, _vp, _vp, _vp, _vp, _sz, _vp]),
    "tcl_score_noalloc_max_bytes": (_sz, []),
    "tcl_score_noalloc": (_i32, [_vp, _i32, _i32, _vp, _vp, _vp, _vp]),
    "tcl_get_params": (_i32, [_vp, _vp, _sz]),
    "tcl_set_params": (_i32, [_vp, _vp, _sz]),
    "tcl_last_error": (ctypes.c_char_p, []),
    "tcl_timing_enable": (_i32, [_vp, _i32]),
    "tcl_timing_count": (_i32, [_vp]),
    "tcl_timing_get": (_i32, [_vp, _i32, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_double),
                              ctypes.POINTER(ctypes.c_int64)]),
    "tcl_timing_reset": (_i32, [_vp]),
    "tcl_trainer_create": (_i32, [_vp, _vp, ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_float,
                                  _i32, _i32, ctypes.POINTER(_vp)]),
    "tcl_trainer_destroy": (_i32, [_vp]),
    "tcl_distill_workspace_bytes": (_sz, [_vp, _i32, _i32]),
    "tcl_distill_step": (_i32, [_vp, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "tcl_trainer_get_grads": (_i32, [_vp, _vp, _sz]),
    "tcl_distill_step_kd": (_i32, [_vp, _i32, _i32, _vp, _vp, _vp, ctypes.POINTER(KDLoss), _vp, _vp, _sz, _vp]),
    "tcl_lambdarank_workspace_bytes": (_sz, [_i32]),
    "tcl_teacher_gate": (_i32, [_i32, _vp, _vp, _vp]),
    "tcl_test_distill_step_kd_ranked": (_i32, [_vp, _i32, _i32, _vp, _vp, _vp, ctypes.POINTER(KDLoss), _vp, _vp,
                                               _vp, _vp, _sz, _vp]),
    "tcl_topk": (_i32, [_i32, _vp, _vp, _i32, _vp, _vp]),
    "tcl_lateral_param_count": (_sz, [ctypes.POINTER(Config), _i32]),
    "tcl_lateral_create": (_i32, [_vp, _vp, _i32, _vp, _sz, ctypes.POINTER(_vp)]),
    "tcl_lateral_destroy": (_i32, [_vp]),
    "tcl_progressive_workspace_bytes": (_sz, [_vp, _i32, _i32]),
    "tcl_progressive_score": (_i32, [_vp, _i32, _i32, _vp, _vp, _vp, _vp, _sz, _vp]),
    "tcl_topk_score_workspace_bytes": (_sz, [_i32, _i32]),
    "tcl_topk_score": (_i32, [_i32, _vp, _vp, _vp, _vp, _i32, _vp, _vp, _sz, _vp]),
    "tcl_rdu_workspace_bytes": (_sz, [_i32, _i32]),
    "tcl_rdu_select": (_i32, [_i32, _vp, _vp, _i32, _vp, _i32, _i32, _vp, _vp, _vp, _sz, _vp]),
    "tcl_lambdarank": (_i32, [_i32, _vp, _vp, ctypes.c_float, _vp, _vp, _vp, _sz, _vp]),
    "tcl_trainer_timing_enable": (_i32, [_vp, _i32]),
    "tcl_trainer_timing_count": (_i32, [_vp]),
    "tcl_trainer_timing_get": (_i32, [_vp, _i32, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_double),
                                      ctypes.POINTER(ctypes.c_int64)]),
    "tcl_trainer_timing_reset": (_i32, [_vp]),
    "tcl_test_gemm_f32": (_i32, [_i32, _i32, _i32, _vp, _vp, _vp, _vp, _i32, _i32, _vp]),
    "tcl_test_gemm_split": (_i32, [_i32, _i32, _i32, _vp, _vp, _i32, _i32, _vp, _vp, _vp, _i32, _i32, _vp, _vp]),
    "tcl_test_gemm_bf16": (_i32, [_i32, _i32, _i32, _i32, _i32, _vp, _vp, _i32, _i32, _vp, _vp, _vp, _vp, _vp]),
    "tcl_test_conv_silu_f32": (_i32, [_i32, _i32, _i32, _vp, _vp, _i32, _vp, _vp, _vp, _vp]),
    "tcl_test_xproj_conv_f32": (_i32, [_i32, _i32, _i32, _i32, _vp, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp,
                                       _vp, _vp]),
    "tcl_test_xproj_conv_bf16": (_i32, [_i32, _i32, _i32, _i32, _vp, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp,
                                        _vp]),
    "tcl_test_offsets": (_i32, [_i32, _i32, _vp, _vp, _vp, _vp]),
    "tcl_test_scan_f32": (_i32, [_i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _i32, _vp, _vp, _vp,
                                 _vp, _vp, _vp]),
}


def lib_path() -> str:
    return _LIB_PATH


def lib():
    """Load libtcl.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with `python -m paper_2604_12891_amd.build`")
        L = ctypes.CDLL(_LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype, fn.argtypes = res, args
        _lib = L
    return _lib


def check(status: int):
    if status != 0:
        raise TclError(status, lib().tcl_last_error().decode())


def make_config(F, d_model, d_inner, d_state, d_conv, dt_rank, n_layers, head_hidden,
                final_norm=1, norm_eps=1e-5, dtype="f32", f32_matmul="split", enc_hidden=(), dec_hidden2=0) -> Config:
    """f32_matmul ("split", "split_bf16" or "native") selects how an fp32 model runs its
    dense projections (tcl_f32_matmul); enc_hidden (up to two widths) and
    dec_hidden2 select the multi-layer encoder and three-layer decoder."""
    enc = list(enc_hidden) + [0] * (2 - len(enc_hidden))
    return Config(F, d_model, d_inner, d_state, d_conv, dt_rank, n_layers, head_hidden, final_norm,
                  norm_eps, TCL_BF16 if dtype == "bf16" else TCL_F32, F32_MATMUL[f32_matmul],
                  (ctypes.c_int32 * 2)(*enc), dec_hidden2)


def config_from_shape(shape, dtype="f32", f32_matmul="split") -> Config:
    return make_config(shape.F, shape.d_model, shape.d_inner, shape.d_state, shape.d_conv, shape.dt_rank,
                       shape.n_layers, shape.head_hidden, shape.final_norm, shape.norm_eps, dtype, f32_matmul,
                       tuple(getattr(shape, "enc_hidden", ())), getattr(shape, "dec_hidden2", 0))


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream=None) -> int:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


class CostModel:
    """A device-resident cost model (tcl_cost_model_create / tcl_score)."""

    def __init__(self, cfg: Config, params: np.ndarray):
        L = lib()
        self.cfg = cfg
        self._n = L.tcl_param_count(ctypes.byref(cfg))
        blob = np.ascontiguousarray(params, dtype=np.float32)
        h = _vp()
        check(L.tcl_cost_model_create(ctypes.byref(cfg), blob.ctypes.data, blob.size, ctypes.byref(h)))
        self._h = h
        self._ws = None

    def close(self):
        if getattr(self, "_h", None):
            check(lib().tcl_cost_model_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def handle(self):
        return self._h

    def workspace_bytes(self, B: int, L: int) -> int:
        return lib().tcl_score_workspace_bytes(self._h, B, L)

    def workspace(self, B: int, L: int):
        import torch
        need = self.workspace_bytes(B, L)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        return self._ws

    def score(self, feats, lengths, out=None, workspace=None, stream=None):
        """feats [B,L,F] fp32 cuda, lengths [B] int32 cuda -> scores [B] fp32 cuda."""
        import torch
        B, L, _ = feats.shape
        if out is None:
            out = torch.empty(B, dtype=torch.float32, device=feats.device)
        ws = self.workspace(B, L) if workspace is None else workspace
        check(lib().tcl_score(self._h, B, L, feats.data_ptr(), lengths.data_ptr(), out.data_ptr(),
                              ws.data_ptr(), ws.numel() * ws.element_size(), _stream(stream)))
        return out

    def score_noalloc(self, feats, lengths, out, stream=None):
        """tcl_score_noalloc: the scores into `out` with the library's own
        scratch buffer (no workspace, nothing allocated)."""
        B, L, _ = feats.shape
        check(lib().tcl_score_noalloc(self._h, B, L, feats.data_ptr(), lengths.data_ptr(), out.data_ptr(),
                                      _stream(stream)))
        return out

    def set_score_streams(self, n: int):
        """1: one pass per batch; 2 (default): batches of >= 2048 programs as
        two concurrent halves (tcl_set_score_streams)."""
        check(lib().tcl_set_score_streams(self._h, n))

    def timing(self, enable: bool):
        check(lib().tcl_timing_enable(self._h, int(enable)))

    def timing_reset(self):
        check(lib().tcl_timing_reset(self._h))

    def timing_report(self) -> dict:
        """{kernel name: (total_ms, launches)} of the launches timed so far."""
        L = lib()
        out = {}
        for i in range(L.tcl_timing_count(self._h)):
            name, ms, n = ctypes.c_char_p(), ctypes.c_double(), ctypes.c_int64()
            check(L.tcl_timing_get(self._h, i, ctypes.byref(name), ctypes.byref(ms), ctypes.byref(n)))
            out[name.value.decode()] = (ms.value, n.value)
        return out

    def get_params(self) -> np.ndarray:
        out = np.empty(self._n, dtype=np.float32)
        check(lib().tcl_get_params(self._h, out.ctypes.data, out.size))
        return out

    def set_params(self, params: np.ndarray):
        blob = np.ascontiguousarray(params, dtype=np.float32)
        check(lib().tcl_set_params(self._h, blob.ctypes.data, blob.size))


class Progressive:
    """A frozen KB and an active column joined by lateral adapters of width
    `adapter` (tcl_lateral_create / tcl_progressive_score). Keeps both models
    alive."""

    def __init__(self, kb: CostModel, ac: CostModel, adapter: int, params: np.ndarray):
        L = lib()
        self.kb, self.ac, self.adapter = kb, ac, adapter
        blob = np.ascontiguousarray(params, dtype=np.float32)
        h = _vp()
        check(L.tcl_lateral_create(kb.handle, ac.handle, adapter, blob.ctypes.data, blob.size, ctypes.byref(h)))
        self._h = h
        self._ws = None

    def close(self):
        if getattr(self, "_h", None):
            check(lib().tcl_lateral_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def workspace(self, B: int, L: int):
        import torch
        need = lib().tcl_progressive_workspace_bytes(self._h, B, L)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        return self._ws

    def score(self, feats, lengths, out=None, workspace=None, stream=None):
        """The AC's scores with the KB read through Eq. (7): feats [B,L,F]
        fp32 cuda, lengths [B] int32 cuda -> [B] fp32 cuda."""
        import torch
        B, L, _ = feats.shape
        if out is None:
            out = torch.empty(B, dtype=torch.float32, device=feats.device)
        ws = self.workspace(B, L) if workspace is None else workspace
        check(lib().tcl_progressive_score(self._h, B, L, feats.data_ptr(), lengths.data_ptr(), out.data_ptr(),
                                          ws.data_ptr(), ws.numel() * ws.element_size(), _stream(stream)))
        return out


class Trainer:
    """Teacher -> student distillation (tcl_trainer_create / tcl_distill_step)."""

    def __init__(self, teacher: CostModel, student: CostModel, lr=1e-3, betas=(0.9, 0.999), eps=1e-8,
                 max_B=1024, max_L=25):
        h = _vp()
        check(lib().tcl_trainer_create(teacher.handle, student.handle, lr, betas[0], betas[1], eps, max_B,
                                       max_L, ctypes.byref(h)))
        self._h = h
        self._n = student._n
        self._keep = (teacher, student)  # the trainer must not outlive its models
        self._ws = None

    def close(self):
        if getattr(self, "_h", None):
            check(lib().tcl_trainer_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def workspace_bytes(self, B: int, L: int) -> int:
        return lib().tcl_distill_workspace_bytes(self._h, B, L)

    def workspace(self, B: int, L: int):
        import torch
        need = self.workspace_bytes(B, L)
        if need == 0:
            raise ValueError(f"B={B}, L={L} exceed the trainer's bounds")
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        return self._ws

    def step(self, feats, lengths, labels, loss=None, workspace=None, stream=None):
        """One step; returns the device tensor [total, mse_teacher, mse_label]."""
        import torch
        B, L, _ = feats.shape
        if loss is None:
            loss = torch.empty(3, dtype=torch.float32, device=feats.device)
        ws = self.workspace(B, L) if workspace is None else workspace
        check(lib().tcl_distill_step(self._h, B, L, feats.data_ptr(), lengths.data_ptr(), labels.data_ptr(),
                                     loss.data_ptr(), ws.data_ptr(), ws.numel() * ws.element_size(),
                                     _stream(stream)))
        return loss

    def step_kd(self, feats, lengths, labels, beta=0.5, phi=1.0, sigma=1.0, ewc_lambda=0.0, fisher=None,
                theta_prev=None, loss=None, workspace=None, stream=None, phi_dev=None, rank_keys=None,
                scores_out=None):
        """One step on the Eq. (9) objective (tcl_distill_step_kd); fisher and
        theta_prev are device fp32 tensors of the parameter count; phi_dev
        (a device fp32 tensor of one element, optional) replaces phi. Returns
        the device tensor [total, rank(s; teacher), rank(s; label), ewc].
        rank_keys / scores_out (device fp32 [B] / [2B]) go through the test
        entry tcl_test_distill_step_kd_ranked."""
        import torch
        B, L, _ = feats.shape
        if loss is None:
            loss = torch.empty(4, dtype=torch.float32, device=feats.device)
        ws = self.workspace(B, L) if workspace is None else workspace
        kd = KDLoss(beta, phi, sigma, ewc_lambda, _ptr(fisher), _ptr(theta_prev), _ptr(phi_dev))
        if rank_keys is None and scores_out is None:
            check(lib().tcl_distill_step_kd(self._h, B, L, feats.data_ptr(), lengths.data_ptr(),
                                            labels.data_ptr(), ctypes.byref(kd), loss.data_ptr(), ws.data_ptr(),
                                            ws.numel() * ws.element_size(), _stream(stream)))
        else:
            check(lib().tcl_test_distill_step_kd_ranked(
                self._h, B, L, feats.data_ptr(), lengths.data_ptr(), labels.data_ptr(), ctypes.byref(kd),
                _ptr(rank_keys), _ptr(scores_out), loss.data_ptr(), ws.data_ptr(), ws.numel() * ws.element_size(),
                _stream(stream)))
        return loss

    def grads(self) -> np.ndarray:
        out = np.empty(self._n, dtype=np.float32)
        check(lib().tcl_trainer_get_grads(self._h, out.ctypes.data, out.size))
        return out

    def timing(self, enable: bool):
        check(lib().tcl_trainer_timing_enable(self._h, int(enable)))

    def timing_reset(self):
        check(lib().tcl_trainer_timing_reset(self._h))

    def timing_report(self) -> dict:
        L = lib()
        out = {}
        for i in range(L.tcl_trainer_timing_count(self._h)):
            name, ms, n = ctypes.c_char_p(), ctypes.c_double(), ctypes.c_int64()
            check(L.tcl_trainer_timing_get(self._h, i, ctypes.byref(name), ctypes.byref(ms), ctypes.byref(n)))
            out[name.value.decode()] = (ms.value, n.value)
        return out


def gemm_f32(A, W, bias=None, out=None, stream=None, tile=-1, epilogue=0):
    """epilogue 0: A W^T (+ bias); 1: out += A W^T; 2: rstd(A) * A W^T."""
    import torch
    M, K = A.shape
    N = W.shape[0]
    if out is None:
        out = torch.empty(M, N, dtype=torch.float32, device=A.device)
    check(lib().tcl_test_gemm_f32(M, N, K, A.data_ptr(), W.data_ptr(), _ptr(bias), out.data_ptr(), tile,
                                  epilogue, _stream(stream)))
    return out


def topk(scores, seg_offsets, K, stream=None):
    """Per-segment top-K (tcl_topk): scores fp32 [n], seg_offsets int32
    [n_seg + 1] (device); returns int32 [n_seg, K] global indices."""
    import torch
    n_seg = seg_offsets.numel() - 1
    out = torch.empty(n_seg, K, dtype=torch.int32, device=scores.device)
    check(lib().tcl_topk(n_seg, seg_offsets.data_ptr(), scores.data_ptr(), K, out.data_ptr(), _stream(stream)))
    return out


def topk_score(scores, latency, weight, seg_offsets, k, stream=None):
    """The Top-k score of Eq. (12) (tcl_topk_score): scores and latency fp32
    [n], weight fp32 [n_seg], seg_offsets int32 [n_seg + 1] (device).
    Returns a device fp64 tensor [3]: Top-k, numerator, denominator."""
    import torch
    n_seg = seg_offsets.numel() - 1
    out = torch.empty(3, dtype=torch.float64, device=scores.device)
    need = lib().tcl_topk_score_workspace_bytes(n_seg, k)
    ws = torch.empty(max(need, 256), dtype=torch.uint8, device=scores.device)
    check(lib().tcl_topk_score(n_seg, seg_offsets.data_ptr(), scores.data_ptr(), latency.data_ptr(),
                               weight.data_ptr(), k, out.data_ptr(), ws.data_ptr(), ws.numel(), _stream(stream)))
    return out


def rdu_select(scores, op, n_ops, initial, n_select, workspace=None, stream=None):
    """RDU selection (tcl_rdu_select): scores fp32 [N], op int32 [N], initial
    int32 [M0] (device). Returns (selected int32 [n_select], count int32 [1])."""
    import torch
    N = scores.numel()
    sel = torch.empty(max(n_select, 1), dtype=torch.int32, device=scores.device)
    cnt = torch.empty(1, dtype=torch.int32, device=scores.device)
    need = lib().tcl_rdu_workspace_bytes(N, n_ops)
    ws = workspace
    if ws is None or ws.numel() * ws.element_size() < need:
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device=scores.device)
    check(lib().tcl_rdu_select(N, scores.data_ptr(), op.data_ptr(), n_ops, initial.data_ptr(), initial.numel(),
                               n_select, sel.data_ptr(), cnt.data_ptr(), ws.data_ptr(),
                               ws.numel() * ws.element_size(), _stream(stream)))
    return sel[:n_select], cnt


def lambdarank(scores, labels, sigma=1.0, grad=True, stream=None):
    """The LambdaRank loss of Eq. (6) (tcl_lambdarank) on device fp32 [B]
    tensors: returns (loss [1], grad [B] or None) as device tensors."""
    import torch
    B = scores.numel()
    loss = torch.empty(1, dtype=torch.float32, device=scores.device)
    g = torch.empty(B, dtype=torch.float32, device=scores.device) if grad else None
    nbytes = lib().tcl_lambdarank_workspace_bytes(B)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=scores.device)
    check(lib().tcl_lambdarank(B, scores.data_ptr(), labels.data_ptr(), sigma, loss.data_ptr(), _ptr(g),
                               ws.data_ptr(), ws.numel(), _stream(stream)))
    return loss, g


def teacher_gate(e, out=None, stream=None):
    """The teacher-loss gate of Eq. (10)-(11) (tcl_teacher_gate) over device
    fp32 batch losses e [n]; returns phi [n] (device)."""
    import torch
    if out is None:
        out = torch.empty_like(e)
    check(lib().tcl_teacher_gate(e.numel(), e.data_ptr(), out.data_ptr(), _stream(stream)))
    return out


def gemm_split(A, W, bias=None, out=None, stream=None, variant=-1, epilogue=0, offs=None):
    """The split-path fp32 GEMM (tcl_test_gemm_split). epilogue 0: A W^T
    (+ bias); 1: out += A W^T; 2: rstd(A) * A W^T; 3: A fp32 [B, L, K]
    gathered by offs [B+1], + bias, out [B*L, N]. variant 1 (32-row panels),
    2 (16-row panels), 3 (32-row panels, all N in registers), 4 (32-row
    panels, K in two halves on two wavefronts per SIMD) or -1."""
    import torch
    N, K = W.shape
    if epilogue == 3:
        Bp, L, _ = A.shape
        M = Bp * L
    else:
        M, Bp, L = A.shape[0], 0, 0
    if out is None:
        if epilogue == 1:
            raise ValueError("epilogue 1 accumulates into out")
        out = torch.empty(M, N, dtype=torch.float32, device=A.device)
    Kw = (K + 7) // 8 * 8
    scratch = torch.empty(3 * N * Kw, dtype=torch.int16, device=A.device)
    check(lib().tcl_test_gemm_split(M, N, K, A.data_ptr(), _ptr(offs), Bp, L, W.data_ptr(), _ptr(bias),
                                    out.data_ptr(), variant, epilogue, scratch.data_ptr(), _stream(stream)))
    return out


(GEMM_BF16_F32, GEMM_BF16_BF16, GEMM_BF16_NORM, GEMM_BF16_RESID, GEMM_BF16_GATHER, GEMM_BF16_F32A,
 GEMM_BF16_F32A_RESID) = range(7)


def gemm_bf16(A, W, bias=None, out=None, stream=None, kind=GEMM_BF16_F32, tile=-1, gain=None, offs=None):
    """The bf16 GEMM variants (see tcl_test_gemm_bf16): W [N, round_up(K, 8)]
    torch.bfloat16, zero-padded in K.
    GEMM_BF16_F32: A bf16 [M,K] -> fp32 (+ bias); GEMM_BF16_BF16: -> bf16;
    GEMM_BF16_NORM: A fp32 -> RMSNorm(gain) -> bf16; GEMM_BF16_RESID: out
    (fp32, required) += A W^T; GEMM_BF16_GATHER: A fp32 [B, L, K] gathered
    by offs [B+1] -> fp32 + bias, out [B*L, N]; GEMM_BF16_F32A: A fp32
    (rounded to bf16) -> fp32; GEMM_BF16_F32A_RESID: out (fp32, required)
    += bf16(A) W^T."""
    import torch
    N = W.shape[0]
    if kind == GEMM_BF16_GATHER:
        Bp, L, K = A.shape
        M = Bp * L
    else:
        (M, K), Bp, L = A.shape, 0, 0
    if W.shape[1] != (K + 7) // 8 * 8:
        raise ValueError(f"W must be [N, {(K + 7) // 8 * 8}] (K zero-padded to a multiple of 8)")
    if out is None:
        if kind in (GEMM_BF16_RESID, GEMM_BF16_F32A_RESID):
            raise ValueError("the residual kinds accumulate into out")
        bf16_out = kind in (GEMM_BF16_BF16, GEMM_BF16_NORM)
        out = torch.empty(M, N, dtype=torch.bfloat16 if bf16_out else torch.float32, device=A.device)
    check(lib().tcl_test_gemm_bf16(kind, tile, M, N, K, A.data_ptr(), _ptr(offs), Bp, L, W.data_ptr(),
                                   _ptr(bias), _ptr(gain), out.data_ptr(), _stream(stream)))
    return out


def conv_silu_f32(offs, x, w, b, E, out, ldx=None, stream=None):
    B = offs.numel() - 1
    check(lib().tcl_test_conv_silu_f32(B, E, w.shape[1], offs.data_ptr(), x.data_ptr(),
                                       x.shape[1] if ldx is None else ldx, w.data_ptr(), b.data_ptr(),
                                       out.data_ptr(), _stream(stream)))
    return out


def xproj_conv_f32(offs, x, w, b, W, rows, E, ldx=None, stream=None):
    """The fused conv + SiLU + x_proj kernel (tcl_test_xproj_conv_f32):
    returns (u [rows, E], xdbl [rows, N]); rows past offs[B] are NaN."""
    import torch
    B = offs.numel() - 1
    N = W.shape[0]
    u = torch.full((rows, E), float("nan"), dtype=torch.float32, device=x.device)
    xdbl = torch.full((rows, N), float("nan"), dtype=torch.float32, device=x.device)
    wsplit = torch.empty(3 * N * E, dtype=torch.int16, device=x.device)
    tpos = torch.empty(rows, dtype=torch.uint8, device=x.device)
    check(lib().tcl_test_xproj_conv_f32(B, rows, E, N, offs.data_ptr(), x.data_ptr(),
                                        x.shape[1] if ldx is None else ldx, w.data_ptr(), b.data_ptr(),
                                        W.data_ptr(), wsplit.data_ptr(), tpos.data_ptr(), u.data_ptr(),
                                        xdbl.data_ptr(), _stream(stream)))
    return u, xdbl


def xproj_conv_bf16(offs, x, w, b, W, rows, E, ldx=None, stream=None):
    """The bf16 fused conv + SiLU + x_proj kernel (tcl_test_xproj_conv_bf16):
    x torch.bfloat16 [rows, ldx], W torch.bfloat16 [N, E]; returns (u bf16
    [rows, E], xdbl fp32 [rows, N]); rows past offs[B] are left as they were
    (u zero, xdbl NaN)."""
    import torch
    B = offs.numel() - 1
    N = W.shape[0]
    u = torch.zeros((rows, E), dtype=torch.bfloat16, device=x.device)
    xdbl = torch.full((rows, N), float("nan"), dtype=torch.float32, device=x.device)
    tpos = torch.empty(rows, dtype=torch.uint8, device=x.device)
    check(lib().tcl_test_xproj_conv_bf16(B, rows, E, N, offs.data_ptr(), x.data_ptr(),
                                         x.shape[1] if ldx is None else ldx, w.data_ptr(), b.data_ptr(),
                                         W.data_ptr(), tpos.data_ptr(), u.data_ptr(), xdbl.data_ptr(),
                                         _stream(stream)))
    return u, xdbl


def offsets(lengths, L, ord=None, stream=None):
    """tcl_test_offsets: returns the device int32 offsets [B+1]; ord (a
    device int32 [B] tensor, optional) receives the longest-first order."""
    import torch
    B = lengths.numel()
    offs = torch.empty(B + 1, dtype=torch.int32, device=lengths.device)
    check(lib().tcl_test_offsets(B, L, lengths.data_ptr(), offs.data_ptr(), _ptr(ord), _stream(stream)))
    return offs


def scan_f32(offs, u, xdbl, z, W_dt, b_dt, A_log, D, out, ldz=None, stream=None, chunks=0):
    """chunks = 0: sequential scan; 1..8: chunked two-level scan."""
    B = offs.numel() - 1
    E = u.shape[1]
    N = A_log.shape[1]
    R = W_dt.shape[1]
    check(lib().tcl_test_scan_f32(B, E, N, R, chunks, offs.data_ptr(), u.data_ptr(), xdbl.data_ptr(), z.data_ptr(),
                                  z.shape[1] if ldz is None else ldz, W_dt.data_ptr(), b_dt.data_ptr(),
                                  A_log.data_ptr(), D.data_ptr(), out.data_ptr(), _stream(stream)))
    return out
