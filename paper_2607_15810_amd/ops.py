"""The library's calls on torch tensors.

torch provides device memory and the current HIP stream; each function
allocates its outputs (and workspace) as torch tensors and hands raw device
pointers to libquads.so.  Nothing here computes any part of the layer.
"""

from dataclasses import dataclass
from typing import Optional

import torch

from . import quads as Q


def _stream():
    return ctypes_void(torch.cuda.current_stream().cuda_stream)


def ctypes_void(v):
    return int(v) if v is not None else None


def _ptr(t):
    return None if t is None else t.data_ptr()


def _require_cuda(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("libquads operates on GPU tensors")


def _ws(nbytes, device):
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


@dataclass
class NVFP4Tensor:
    """codes uint8 [G][R][C/2], scales uint8 [G][R][C/16], gscale f32 [G][2];
    scales_frag: None, or the scales in fragment order (weights only)."""
    codes: torch.Tensor
    scales: torch.Tensor
    gscale: torch.Tensor
    groups: int
    rows: int
    cols: int
    scales_frag: Optional[torch.Tensor] = None

    @staticmethod
    def empty(groups, rows, cols, device):
        return NVFP4Tensor(
            torch.empty((groups, rows, cols // 2), dtype=torch.uint8, device=device),
            torch.empty((groups, rows, cols // 16), dtype=torch.uint8, device=device),
            torch.empty((groups, 2), dtype=torch.float32, device=device),
            groups, rows, cols)

    def struct(self):
        return Q.NVFP4(self.codes.data_ptr(), self.scales.data_ptr(), self.gscale.data_ptr(),
                       self.groups, self.rows, self.cols,
                       self.scales_frag.data_ptr() if self.scales_frag is not None else None)

    def ref(self):
        import ctypes
        s = self.struct()
        self._keep = s
        return ctypes.byref(s)


def _nv(t):
    if t is None:
        return None
    import ctypes
    s = t.struct()
    return ctypes.pointer(s)


def quantize_act(x, amax_partials=None, rac=False):
    """Q_A of x ([rows][cols] bf16 or f32).  With rac=True also returns the
    fused RAC channel scores (uint64 as int64 tensor) and max|r| (float [1])."""
    _require_cuda(x)
    x = x.contiguous()
    rows, cols = x.shape
    dt = Q.QD_DTYPE_BF16 if x.dtype == torch.bfloat16 else Q.QD_DTYPE_F32
    out = NVFP4Tensor.empty(1, rows, cols, x.device)
    ws = _ws(Q.lib().nvfp4_quantize_act_workspace(rows, cols), x.device)
    scores = ramax = None
    if rac:
        scores = torch.empty(cols, dtype=torch.int64, device=x.device)
        ramax = torch.empty(1, dtype=torch.float32, device=x.device)
    n_part = 0 if amax_partials is None else amax_partials.numel()
    Q.call("nvfp4_quantize_act", x.data_ptr(), dt, rows, cols, _ptr(amax_partials), n_part,
           _nv(out), _ptr(scores), _ptr(ramax), ws.data_ptr(), ws.numel(), _stream())
    return out, scores, ramax


def quantize_weight(w, frag_scales=True):
    """Q_W of a bf16 bank [groups][rows][cols], one tensor scale per group.
    With frag_scales (and rows % 16 == 0, cols % 256 == 0) the result also
    carries the fragment-ordered copy of its scales (pack_frag_scales)."""
    _require_cuda(w)
    w = w.contiguous()
    if w.dim() == 2:
        w = w.unsqueeze(0)
    G, R, C = w.shape
    out = NVFP4Tensor.empty(G, R, C, w.device)
    ws = _ws(Q.lib().nvfp4_quantize_weight_workspace(G, R, C), w.device)
    Q.call("nvfp4_quantize_weight", w.data_ptr(), G, R, C, _nv(out), ws.data_ptr(), ws.numel(),
           _stream())
    if frag_scales and Q.lib().nvfp4_frag_scales_bytes(G, R, C) > 0:
        out.scales_frag = pack_frag_scales(out)
    return out


def pack_frag_scales(t):
    """The scales of weight tensor t re-laid out in fragment order: uint8
    [G][R/16][C/256][256] (nvfp4_pack_frag_scales)."""
    n = Q.lib().nvfp4_frag_scales_bytes(t.groups, t.rows, t.cols)
    if n <= 0:
        raise ValueError("fragment-ordered scales need rows % 16 == 0 and cols % 256 == 0")
    out = torch.empty((t.groups, t.rows // 16, t.cols // 256, 256), dtype=torch.uint8,
                      device=t.codes.device)
    plain = NVFP4Tensor(t.codes, t.scales, t.gscale, t.groups, t.rows, t.cols)
    Q.call("nvfp4_pack_frag_scales", _nv(plain), out.data_ptr(), _stream())
    return out


def dequantize(t, unscaled=False, dtype=torch.float32):
    out = torch.empty((t.groups, t.rows, t.cols), dtype=dtype, device=t.codes.device)
    dt = Q.QD_DTYPE_BF16 if dtype == torch.bfloat16 else Q.QD_DTYPE_F32
    Q.call("nvfp4_dequantize", _nv(t), int(unscaled), out.data_ptr(), dt, _stream())
    return out


def route_permute(logits, k, renorm=True):
    _require_cuda(logits)
    logits = logits.contiguous().float()
    T, E = logits.shape
    dev = logits.device
    ids = torch.empty((T, k), dtype=torch.int32, device=dev)
    w = torch.empty((T, k), dtype=torch.float32, device=dev)
    offs = torch.empty(E + 1, dtype=torch.int32, device=dev)
    row_token = torch.empty(max(T * k, 1), dtype=torch.int32, device=dev)
    inv_row = torch.empty((T, k), dtype=torch.int32, device=dev)
    ws = _ws(Q.lib().moe_route_permute_workspace(T, E, k), dev)
    Q.call("moe_route_permute", logits.data_ptr(), T, E, k, int(renorm), ids.data_ptr(),
           w.data_ptr(), offs.data_ptr(), row_token.data_ptr(), inv_row.data_ptr(),
           ws.data_ptr(), ws.numel(), _stream())
    return ids, w, offs, row_token[:T * k], inv_row


def select_channels(x, xq, Ks, scores=None, ramax=None):
    """RAC selection + masked residual.  scores/ramax from quantize_act(rac=True)
    are used as given; otherwise they are computed here."""
    _require_cuda(x)
    T, K = x.shape
    dev = x.device
    ready = scores is not None
    if not ready:
        scores = torch.empty(K, dtype=torch.int64, device=dev)
        ramax = torch.empty(1, dtype=torch.float32, device=dev)
    sel = torch.empty(max(Ks, 1), dtype=torch.int32, device=dev)
    rq = NVFP4Tensor.empty(1, T, K, dev)
    ws = _ws(Q.lib().rac_select_channels_workspace(T, K), dev)
    Q.call("rac_select_channels", x.data_ptr(), _nv(xq), Ks, scores.data_ptr(), ramax.data_ptr(),
           int(ready), sel.data_ptr(), _nv(rq), ws.data_ptr(), ws.numel(), _stream())
    return sel[:Ks], rq, scores, ramax


def select_channels_per_expert(x, xq, Ks, row_token, offsets):
    """Per-expert RAC sets over the permuted rows (row_token, offsets from
    route_permute): returns (sel_pe [E][Ks], rq (all channels), rq_rows
    [rows][width] f16, scores_pe [E][K] as int64, ramax [1])."""
    _require_cuda(x)
    T, K = x.shape
    dev = x.device
    E = int(offsets.numel()) - 1
    rows = int(row_token.numel())
    scores = torch.empty((E, K), dtype=torch.int64, device=dev)
    ramax = torch.empty(1, dtype=torch.float32, device=dev)
    sel = torch.empty((E, max(Ks, 1)), dtype=torch.int32, device=dev)
    rq = NVFP4Tensor.empty(1, T, K, dev)
    width = Q.lib().rac_selected_width(Ks)
    rows_out = torch.empty((max(rows, 1), max(width, 8)), dtype=torch.float16, device=dev)
    ws = _ws(Q.lib().rac_select_channels_per_expert_workspace(T, K, E), dev)
    Q.call("rac_select_channels_per_expert", x.data_ptr(), _nv(xq), Ks, row_token.data_ptr(),
           offsets.data_ptr(), E, rows, scores.data_ptr(), ramax.data_ptr(), sel.data_ptr(),
           _nv(rq), rows_out.data_ptr(), ws.data_ptr(), ws.numel(), _stream())
    return sel[:, :Ks], rq, rows_out[:rows, :width], scores, ramax


def grouped_gemm_per_expert(a, w, rows, row_token, offsets, rq, sel_pe, rq_rows,
                            epilogue=Q.QD_EPI_NONE, want_amax=False):
    """The grouped GEMM with one RAC channel set per expert (sel_pe [E][Ks],
    rq_rows from select_channels_per_expert)."""
    dev = a.codes.device
    E, N, Ks = w.groups, w.rows, int(sel_pe.shape[1])
    ncol = N // 2 if epilogue == Q.QD_EPI_SWIGLU else N
    out = torch.empty((rows, ncol), dtype=torch.bfloat16, device=dev)
    amax = None
    if want_amax:
        cnt = Q.lib().moe_w4a4_grouped_gemm_per_expert_amax_count(rows, N, a.cols, E, Ks, epilogue)
        amax = torch.empty(max(cnt, 1), dtype=torch.float32, device=dev)
    sel_c = sel_pe.contiguous()
    rr = rq_rows.contiguous()
    Q.call("moe_w4a4_grouped_gemm_per_expert", _nv(a), _ptr(row_token), offsets.data_ptr(), E,
           rows, _nv(w), _nv(rq), sel_c.data_ptr(), Ks, rr.data_ptr(), epilogue, out.data_ptr(),
           _ptr(amax), _stream())
    return out, amax


def gather_selected(rq, sel):
    """The masked residual at the selected channels, compacted per row: f16
    [rows][rac_selected_width(Ks)] (no tensor scale; zero past Ks)."""
    Ks = int(sel.numel())
    width = Q.lib().rac_selected_width(Ks)
    out = torch.empty((rq.rows, max(width, 8)), dtype=torch.float16, device=rq.codes.device)
    Q.call("rac_gather_selected", _nv(rq), _ptr(sel), Ks, out.data_ptr(), _stream())
    return out[:, :width]


def residual_gemm(rq, sel, w, rows, row_token=None, offsets=None):
    dev = rq.codes.device
    out = torch.empty((rows, w.rows), dtype=torch.float32, device=dev)
    Q.call("rac_residual_gemm", _nv(rq), _ptr(sel), int(sel.numel()), _ptr(row_token),
           _ptr(offsets), rows, _nv(w), out.data_ptr(), _stream())
    return out


def grouped_gemm(a, w, rows, row_token=None, offsets=None, rq=None, sel=None,
                 epilogue=Q.QD_EPI_NONE, want_amax=False, rq_sel=None):
    """rq_sel: the compact residual (gather_selected(rq, sel)); formed here
    when the kernel for these sizes reads it and it is not given."""
    dev = a.codes.device
    E = w.groups
    N = w.rows
    ncol = N // 2 if epilogue == Q.QD_EPI_SWIGLU else N
    out = torch.empty((rows, ncol), dtype=torch.bfloat16, device=dev)
    amax = None
    Ks = 0 if sel is None else int(sel.numel())
    if want_amax:
        cnt = Q.lib().moe_w4a4_grouped_gemm_amax_count(rows, N, a.cols, E, Ks, epilogue)
        amax = torch.empty(max(cnt, 1), dtype=torch.float32, device=dev)
    if Ks and rq_sel is None and Q.lib().moe_w4a4_grouped_gemm_residual_form(
            rows, N, a.cols, E, Ks, epilogue) == 2:
        rq_sel = gather_selected(rq, sel)
    Q.call("moe_w4a4_grouped_gemm", _nv(a), _ptr(row_token), _ptr(offsets), E, rows, _nv(w),
           _nv(rq) if Ks else None, _ptr(sel) if Ks else None, Ks,
           _ptr(rq_sel) if Ks else None, epilogue, out.data_ptr(), _ptr(amax), _stream())
    return out, amax


def unpermute_combine(z, inv_row, w):
    T, k = inv_row.shape
    H = z.shape[1]
    y = torch.empty((T, H), dtype=torch.bfloat16, device=z.device)
    Q.call("moe_unpermute_combine", z.data_ptr(), inv_row.data_ptr(), w.data_ptr(), T, k, H,
           y.data_ptr(), _stream())
    return y


class MoELayer:
    """The whole layer through qd_moe_layer_forward, with a reusable
    workspace; `views()` exposes the intermediates of the last call."""

    def __init__(self, w13, w2, T, k, Ks, renorm=True, ws=None, Ks2=0):
        """Ks: channels compensated at the W13 input; Ks2: at the W2 input."""
        self.w13, self.w2 = w13, w2
        self.E = w13.groups
        self.I = w13.rows // 2
        self.H = w13.cols
        self.T, self.k, self.Ks, self.Ks2, self.renorm = T, k, Ks, Ks2, renorm
        dev = w13.codes.device
        n = Q.lib().qd_moe_layer_workspace(T, self.H, self.E, k, self.I)
        self.ws = _ws(n, dev) if ws is None else ws
        if self.ws.numel() < n:
            raise ValueError("workspace too small")
        import ctypes
        off = (ctypes.c_int64 * len(Q.VIEW_NAMES))()
        Q.call("qd_moe_layer_views", T, self.H, self.E, k, self.I, off)
        self.off = list(off)
        self._s13 = w13.struct()
        self._s2 = w2.struct()

    def __call__(self, x, logits, y=None, events=None):
        """events: optional list of QD_STAGE_COUNT + 1 recorded torch.cuda.Event
        objects (enable_timing=True); they are re-recorded at the stage
        boundaries on the current stream."""
        import ctypes
        if y is None:
            y = torch.empty((self.T, self.H), dtype=torch.bfloat16, device=x.device)
        evp = None
        if events is not None:
            evp = (ctypes.c_void_p * len(events))(*[e.cuda_event for e in events])
        Q.call("qd_moe_layer_forward_timed", x.data_ptr(), logits.data_ptr(), self.T, self.H,
               self.E, self.k, self.I, self.Ks, self.Ks2, int(self.renorm),
               ctypes.byref(self._s13), ctypes.byref(self._s2), y.data_ptr(),
               self.ws.data_ptr(), self.ws.numel(), evp, _stream())
        return y

    def view(self, name, dtype, shape):
        i = Q.VIEW_NAMES.index(name)
        nbytes = 1
        for s in shape:
            nbytes *= s
        nbytes *= torch.tensor([], dtype=dtype).element_size()
        start = self.off[i]
        return self.ws[start:start + nbytes].view(dtype).view(*shape)

    def views(self):
        T, H, E, k, I = self.T, self.H, self.E, self.k, self.I
        R = T * k
        u8, i32, f32 = torch.uint8, torch.int32, torch.float32
        return dict(
            ids=self.view("topk_ids", i32, (T, k)), w=self.view("topk_w", f32, (T, k)),
            offsets=self.view("offsets", i32, (E + 1,)),
            row_token=self.view("row_token", i32, (R,)),
            inv_row=self.view("inv_row", i32, (T, k)),
            xq_codes=self.view("xq_codes", u8, (T, H // 2)),
            xq_scales=self.view("xq_scales", u8, (T, H // 16)),
            xq_gscale=self.view("xq_gscale", f32, (2,)),
            scores=self.view("scores", torch.int64, (H,)),
            ramax=self.view("ramax", f32, (1,)),
            sel=self.view("sel", i32, (self.Ks,)),
            rq_codes=self.view("rq_codes", u8, (T, H // 2)),
            rq_scales=self.view("rq_scales", u8, (T, H // 16)),
            rq_gscale=self.view("rq_gscale", f32, (2,)),
            h=self.view("h", torch.bfloat16, (R, I)),
            hq_codes=self.view("hq_codes", u8, (R, I // 2)),
            hq_scales=self.view("hq_scales", u8, (R, I // 16)),
            hq_gscale=self.view("hq_gscale", f32, (2,)),
            z=self.view("z", torch.bfloat16, (R, H)),
            rq_sel=self.view("rq_sel", torch.float16, (T, Q.lib().rac_selected_width(self.Ks))),
            h_scores=self.view("h_scores", torch.int64, (I,)),
            h_ramax=self.view("h_ramax", f32, (1,)),
            sel2=self.view("sel2", i32, (self.Ks2,)),
            hr_codes=self.view("hr_codes", u8, (R, I // 2)),
            hr_scales=self.view("hr_scales", u8, (R, I // 16)),
            hr_gscale=self.view("hr_gscale", f32, (2,)),
            hr_sel=self.view("hr_sel", torch.float16,
                             (R, Q.lib().rac_selected_width(self.Ks2))),
        )


class MoEBlock(MoELayer):
    """The layer fed from the hidden state through qd_moe_block_forward:
    RMSNorm (gamma, eps) and the router (w_router [E][H] bf16) folded into
    the layer's first launch; `views()` adds x (the normalised state) and the
    router logits."""

    def __init__(self, w13, w2, T, k, Ks, gamma, w_router, eps=1e-6, renorm=True, Ks2=0):
        import ctypes
        self.w13, self.w2 = w13, w2
        self.E = w13.groups
        self.I = w13.rows // 2
        self.H = w13.cols
        self.T, self.k, self.Ks, self.Ks2, self.renorm = T, k, Ks, Ks2, renorm
        _require_cuda(gamma, w_router)
        if gamma.dtype != torch.bfloat16 or w_router.dtype != torch.bfloat16:
            raise TypeError("gamma and w_router must be bfloat16")
        self.gamma = gamma.contiguous()
        self.w_router = w_router.contiguous()
        self.eps = float(eps)
        n = Q.lib().qd_moe_block_workspace(T, self.H, self.E, k, self.I)
        self.ws = _ws(n, w13.codes.device)
        off = (ctypes.c_int64 * (len(Q.VIEW_NAMES) + 2))()
        Q.call("qd_moe_block_views", T, self.H, self.E, k, self.I, off)
        self.off = list(off)
        self._s13 = w13.struct()
        self._s2 = w2.struct()

    def __call__(self, h, y=None, events=None):
        import ctypes
        _require_cuda(h)
        if h.dtype != torch.bfloat16:
            raise TypeError("h must be bfloat16")
        h = h.contiguous()
        if y is None:
            y = torch.empty((self.T, self.H), dtype=torch.bfloat16, device=h.device)
        evp = None
        if events is not None:
            evp = (ctypes.c_void_p * len(events))(*[e.cuda_event for e in events])
        Q.call("qd_moe_block_forward_timed", h.data_ptr(), self.gamma.data_ptr(), self.eps,
               self.w_router.data_ptr(), self.T, self.H, self.E, self.k, self.I, self.Ks,
               self.Ks2, int(self.renorm), ctypes.byref(self._s13), ctypes.byref(self._s2),
               y.data_ptr(), self.ws.data_ptr(), self.ws.numel(), evp, _stream())
        return y

    def views(self):
        v = super().views()
        n = len(Q.VIEW_NAMES)
        T, H, E = self.T, self.H, self.E
        v["x"] = self.ws[self.off[n]:self.off[n] + T * H * 2].view(torch.bfloat16).view(T, H)
        v["logits"] = self.ws[self.off[n + 1]:self.off[n + 1] + T * E * 4].view(
            torch.float32).view(T, E)
        return v


class MoELayerPerExpert:
    """The layer with one RAC channel set per expert at the W13 input
    (qd_moe_layer_forward_per_expert), with a reusable workspace."""

    def __init__(self, w13, w2, T, k, Ks, renorm=True):
        self.w13, self.w2 = w13, w2
        self.E = w13.groups
        self.I = w13.rows // 2
        self.H = w13.cols
        self.T, self.k, self.Ks, self.renorm = T, k, Ks, renorm
        n = Q.lib().qd_moe_layer_per_expert_workspace(T, self.H, self.E, k, self.I, Ks)
        self.ws = _ws(n, w13.codes.device)
        self._s13 = w13.struct()
        self._s2 = w2.struct()

    def __call__(self, x, logits, y=None):
        import ctypes
        if y is None:
            y = torch.empty((self.T, self.H), dtype=torch.bfloat16, device=x.device)
        Q.call("qd_moe_layer_forward_per_expert", x.data_ptr(), logits.data_ptr(), self.T,
               self.H, self.E, self.k, self.I, self.Ks, int(self.renorm),
               ctypes.byref(self._s13), ctypes.byref(self._s2), y.data_ptr(),
               self.ws.data_ptr(), self.ws.numel(), _stream())
        return y


# ---------------------------------------------------------------- W4A16 (trainer-side forward)

def w4a16_grouped_gemm(a, w, rows, row_token=None, offsets=None, epilogue=Q.QD_EPI_NONE):
    """bf16 activations a [a_rows][K] times the NVFP4 weights w (E groups of
    [N][K]) through moe_w4a16_grouped_gemm."""
    _require_cuda(a)
    a = a.contiguous()
    if a.dtype != torch.bfloat16:
        raise TypeError("a must be bfloat16")
    N = w.rows
    ncol = N // 2 if epilogue == Q.QD_EPI_SWIGLU else N
    out = torch.empty((rows, ncol), dtype=torch.bfloat16, device=a.device)
    Q.call("moe_w4a16_grouped_gemm", a.data_ptr(), a.shape[0], _ptr(row_token), _ptr(offsets),
           w.groups, rows, _nv(w), epilogue, out.data_ptr(), _stream())
    return out


class W4A16MoELayer:
    """The layer's forward with bf16 activations and the fake-quantised
    weights (the trainer side of Sec. 3.2): routing, W13 with SwiGLU, W2 and
    the combine, every step on the library's kernels."""

    def __init__(self, w13, w2, k, renorm=True):
        self.w13, self.w2, self.k, self.renorm = w13, w2, k, renorm

    def __call__(self, x, logits):
        T = x.shape[0]
        ids, wts, offs, row_token, inv_row = route_permute(logits, self.k, self.renorm)
        R = T * self.k
        h = w4a16_grouped_gemm(x, self.w13, R, row_token, offs, Q.QD_EPI_SWIGLU)
        z = w4a16_grouped_gemm(h, self.w2, R, None, offs)
        return unpermute_combine(z, inv_row, wts)


# ---------------------------------------------------------------- FP8 W8A8 comparison layer

def fp8_quantize_rows(x):
    """E4M3 codes with one f32 scale per row of x ([rows][cols] bf16 or f32;
    a weight bank [E][N][K] is E*N rows).  Returns (codes u8, dec f32)."""
    _require_cuda(x)
    x = x.contiguous()
    cols = x.shape[-1]
    rows = x.numel() // cols if cols else 0
    codes = torch.empty(x.shape, dtype=torch.uint8, device=x.device)
    dec = torch.empty(x.shape[:-1], dtype=torch.float32, device=x.device)
    dt = Q.QD_DTYPE_BF16 if x.dtype == torch.bfloat16 else Q.QD_DTYPE_F32
    Q.call("fp8_quantize_rows", x.data_ptr(), dt, rows, cols, codes.data_ptr(), dec.data_ptr(),
           _stream())
    return codes, dec


def fp8_grouped_gemm(a_codes, a_dec, w_codes, w_dec, rows, row_token=None, offsets=None,
                     epilogue=Q.QD_EPI_NONE):
    E, N, K = w_codes.shape
    ncol = N // 2 if epilogue == Q.QD_EPI_SWIGLU else N
    out = torch.empty((rows, ncol), dtype=torch.bfloat16, device=a_codes.device)
    Q.call("moe_fp8_grouped_gemm", a_codes.data_ptr(), a_dec.data_ptr(), a_codes.shape[0],
           _ptr(row_token), _ptr(offsets), E, rows, w_codes.data_ptr(), w_dec.data_ptr(), N, K,
           epilogue, out.data_ptr(), _stream())
    return out


class FP8MoELayer:
    """The FP8 W8A8 layer through qd_fp8_moe_layer_forward (the comparison
    baseline: same routing, SwiGLU and combine, no residual)."""

    def __init__(self, w13_codes, w13_dec, w2_codes, w2_dec, T, k, renorm=True):
        self.w13 = (w13_codes, w13_dec)
        self.w2 = (w2_codes, w2_dec)
        self.E, N13, self.H = w13_codes.shape
        self.I = N13 // 2
        self.T, self.k, self.renorm = T, k, renorm
        n = Q.lib().qd_fp8_moe_layer_workspace(T, self.H, self.E, k, self.I)
        self.ws = _ws(n, w13_codes.device)

    def __call__(self, x, logits, y=None):
        if y is None:
            y = torch.empty((self.T, self.H), dtype=torch.bfloat16, device=x.device)
        Q.call("qd_fp8_moe_layer_forward", x.data_ptr(), logits.data_ptr(), self.T, self.H,
               self.E, self.k, self.I, int(self.renorm), self.w13[0].data_ptr(),
               self.w13[1].data_ptr(), self.w2[0].data_ptr(), self.w2[1].data_ptr(),
               y.data_ptr(), self.ws.data_ptr(), self.ws.numel(), _stream())
        return y


def mxfp4_quantize_rows(x):
    """MXFP4 codes and E8M0 block scales of x ([..][cols] bf16 or f32,
    cols % 32 == 0; a weight bank [E][N][K] is E*N rows).  Returns
    (codes u8 [..][cols/2], scales u8 [..][cols/32])."""
    _require_cuda(x)
    x = x.contiguous()
    cols = x.shape[-1]
    rows = x.numel() // cols if cols else 0
    codes = torch.empty(x.shape[:-1] + (cols // 2,), dtype=torch.uint8, device=x.device)
    scales = torch.empty(x.shape[:-1] + (cols // 32,), dtype=torch.uint8, device=x.device)
    dt = Q.QD_DTYPE_BF16 if x.dtype == torch.bfloat16 else Q.QD_DTYPE_F32
    Q.call("mxfp4_quantize_rows", x.data_ptr(), dt, rows, cols, codes.data_ptr(),
           scales.data_ptr(), _stream())
    return codes, scales


def mxfp4_grouped_gemm(a_codes, a_scales, w_codes, w_scales, rows, row_token=None, offsets=None,
                       epilogue=Q.QD_EPI_NONE):
    E, N, K2 = w_codes.shape
    K = 2 * K2
    ncol = N // 2 if epilogue == Q.QD_EPI_SWIGLU else N
    out = torch.empty((rows, ncol), dtype=torch.bfloat16, device=a_codes.device)
    Q.call("moe_mxfp4_grouped_gemm", a_codes.data_ptr(), a_scales.data_ptr(), a_codes.shape[0],
           _ptr(row_token), _ptr(offsets), E, rows, w_codes.data_ptr(), w_scales.data_ptr(), N,
           K, epilogue, out.data_ptr(), _stream())
    return out


class MXFP4MoELayer:
    """The MXFP4 W4A4 comparison layer through qd_mxfp4_moe_layer_forward
    (same routing, SwiGLU and combine, no residual)."""

    def __init__(self, w13_codes, w13_scales, w2_codes, w2_scales, T, k, renorm=True):
        self.w13 = (w13_codes, w13_scales)
        self.w2 = (w2_codes, w2_scales)
        self.E, N13, H2 = w13_codes.shape
        self.H = 2 * H2
        self.I = N13 // 2
        self.T, self.k, self.renorm = T, k, renorm
        n = Q.lib().qd_mxfp4_moe_layer_workspace(T, self.H, self.E, k, self.I)
        self.ws = _ws(n, w13_codes.device)

    def __call__(self, x, logits, y=None):
        if y is None:
            y = torch.empty((self.T, self.H), dtype=torch.bfloat16, device=x.device)
        Q.call("qd_mxfp4_moe_layer_forward", x.data_ptr(), logits.data_ptr(), self.T, self.H,
               self.E, self.k, self.I, int(self.renorm), self.w13[0].data_ptr(),
               self.w13[1].data_ptr(), self.w2[0].data_ptr(), self.w2[1].data_ptr(),
               y.data_ptr(), self.ws.data_ptr(), self.ws.numel(), _stream())
        return y

