"""Python-side plan object over the C ABI (argument marshalling only).

torch supplies device memory and the stream; every step of the run happens
in libdycl.so.  ``Plan.run`` takes device tensors; ``run_numpy`` is a
convenience for tests and tools that copies host arrays in and out.
"""

from __future__ import annotations

import ctypes as C

import numpy as np
import torch

from . import _lib
from .lowering import lower_json

check = _lib.check
lib = _lib.lib


HOST_MODES = {"sync": 0, "device": 1, "graph": 2, "persistent": 3}


class Plan:
    def __init__(self, spec_json: str, blob: bytes, max_batch: int, device: int = 0):
        self._h = C.c_void_p()
        self._blob = C.create_string_buffer(blob, len(blob))
        check(lib.dycl_plan_create(spec_json.encode(), C.cast(self._blob, C.c_void_p), len(blob), int(max_batch),
                                   int(device), C.byref(self._h)))
        self.device = device
        self.max_batch = max_batch
        info = self.info()
        self.n_out = int(info["n_out"])
        self.decisions = int(info["decisions"])
        self.aux = bool(info["aux"])
        self.max_len = int(info.get("max_len", 0))   # tokens per sample (a decoding plan), else 0

    @classmethod
    def from_workload(cls, wl, max_batch: int, device: int = 0):
        blob, man = wl.blob()
        return cls(lower_json(wl.arch, man), blob, max_batch, device)

    def close(self):
        if self._h:
            lib.dycl_plan_destroy(self._h)
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def info(self) -> dict:
        keys = ["n_out", "in_bytes", "decisions", "workspace_bytes", "weight_bytes", "max_batch", "aux", "nodes",
                "host_mode", "graph_captures", "max_len"]
        buf = (C.c_int64 * len(keys))()
        n = check(lib.dycl_plan_info(self._h, buf, len(keys)))
        return {k: int(buf[i]) for i, k in enumerate(keys[:n])}

    def set_host_mode(self, mode: str) -> str:
        """'sync' (read the branch counts back at each decision), 'device'
        (counts stay on the device, count-guarded launches), 'graph'
        (device mode replayed from a captured HIP graph) or 'persistent'
        (device mode with a bounded halting loop in one launch); returns the
        previous mode."""
        if mode not in HOST_MODES:
            raise ValueError(f"host mode must be one of {sorted(HOST_MODES)}")
        prev = check(lib.dycl_plan_set_host_mode(self._h, HOST_MODES[mode]))
        return {v: k for k, v in HOST_MODES.items()}[prev]

    def run(self, x: torch.Tensor, aux, logits: torch.Tensor, records: torch.Tensor, stream=None, tokens=None):
        """x, aux, logits (fp32 [B, n_out]) and records (int32 [B, 4]) are
        device tensors; a decoding plan also takes tokens (int32 [B, max_len])."""
        B = x.shape[0]
        if stream is None:
            stream = torch.cuda.current_stream(x.device)
        args = [self._h, C.c_void_p(x.data_ptr()), int(B), C.c_void_p(aux.data_ptr()) if aux is not None else None,
                C.c_void_p(logits.data_ptr()), C.c_void_p(records.data_ptr())]
        if self.max_len:
            check(lib.dycl_run_seq(*args, C.c_void_p(tokens.data_ptr()) if tokens is not None else None,
                                   C.c_void_p(stream.cuda_stream)))
        else:
            check(lib.dycl_run(*args, C.c_void_p(stream.cuda_stream)))

    def outputs(self, B: int, device="cuda"):
        """Fresh (logits, records, tokens) device tensors for a batch of B
        (tokens None for a plan that emits none)."""
        logits = torch.full((max(B, 1), self.n_out), float("nan"), dtype=torch.float32, device=device)
        rec = torch.zeros((max(B, 1), 4), dtype=torch.int32, device=device)
        tok = torch.zeros((max(B, 1), self.max_len), dtype=torch.int32, device=device) if self.max_len else None
        return logits, rec, tok

    def counts(self):
        buf = (C.c_int32 * (2 * max(1, self.decisions)))()
        d = check(lib.dycl_last_counts(self._h, buf, 2 * max(1, self.decisions)))
        return [(int(buf[2 * i]), int(buf[2 * i + 1])) for i in range(d)]

    def profile(self, on: bool):
        check(lib.dycl_profile_enable(self._h, 1 if on else 0))

    def profile_read(self) -> dict:
        rows = (C.c_double * (4 * 16))()
        n = check(lib.dycl_profile_read(self._h, rows, 16))
        out = {}
        for c in range(n):
            name = lib.dycl_profile_class(c).decode()
            out[name] = {"launches": rows[4 * c], "ms": rows[4 * c + 1], "flops": rows[4 * c + 2],
                         "bytes": rows[4 * c + 3]}
        return out

    def profile_launches(self) -> list:
        """Every launch of the last profiled run: class, ms, flops, bytes."""
        n = check(lib.dycl_profile_launches(self._h, None, 0))
        rows = (C.c_double * (4 * max(n, 1)))()
        n = min(n, check(lib.dycl_profile_launches(self._h, rows, n)))
        return [{"class": lib.dycl_profile_class(int(rows[4 * i])).decode(), "ms": rows[4 * i + 1],
                 "flops": rows[4 * i + 2], "bytes": rows[4 * i + 3],
                 "label": lib.dycl_profile_launch_label(self._h, i).decode()} for i in range(n)]


def decode_records(rec: np.ndarray):
    """int32 [B, 4] -> (exit_index, iterations, skip_mask)."""
    rec = np.ascontiguousarray(rec, dtype=np.int32)
    exit_index = rec[:, 0].copy()
    iterations = rec[:, 1].copy()
    skip = rec[:, 2:4].copy().view(np.uint64).reshape(-1)
    return exit_index, iterations, skip


def device_inputs(wl, x: np.ndarray, aux, device="cuda"):
    if x.dtype == np.uint16:
        xt = torch.from_numpy(x.view(np.int16).copy()).view(torch.bfloat16).to(device)
    else:
        xt = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(device)
    at = torch.from_numpy(np.ascontiguousarray(aux, dtype=np.float32)).to(device) if aux is not None else None
    return xt, at


def run_numpy(plan: Plan, wl, x: np.ndarray, aux=None, device="cuda"):
    """Run host arrays through the plan; returns a dict like the oracle's."""
    B = x.shape[0]
    xt, at = device_inputs(wl, x, aux, device)
    logits, rec, tok = plan.outputs(B, device)
    plan.run(xt, at, logits, rec, tokens=tok)
    torch.cuda.synchronize()
    ex, it, sk = decode_records(rec[:B].cpu().numpy())
    out = {"logits": logits[:B].cpu().numpy(), "exit_index": ex, "iterations": it, "skip_mask": sk,
           "counts": plan.counts()}
    if tok is not None:
        out["tokens"] = tok[:B].cpu().numpy()
    return out


def pack_conv_weights(w_bits: np.ndarray) -> np.ndarray:
    """Packed kernel layout (dycl_op_conv_pack) of bf16 weights given as
    uint16 bits [cout][k][k][cin]; returns uint16 host array."""
    cout, k, _, cin = w_bits.shape
    nbytes = lib.dycl_op_conv_packed_bytes(cout, k, cin)
    if nbytes == 0:
        raise ValueError(f"unsupported conv shape {w_bits.shape}")
    w = np.ascontiguousarray(w_bits, dtype=np.uint16)
    out = np.zeros(nbytes // 2, dtype=np.uint16)
    check(lib.dycl_op_conv_pack(w.ctypes.data, cout, k, cin, out.ctypes.data, nbytes))
    return out


def conv_workspace_bytes(n: int, H: int, W: int, cin: int, cout: int, k: int, stride: int, pad: int) -> int:
    return int(lib.dycl_op_conv_workspace_bytes(n, H, W, cin, cout, k, stride, pad))


def conv_maxpool(x: torch.Tensor, packed: torch.Tensor, cout: int, k: int, stride: int, pad: int, scale=None,
                 shift=None, act: int = 1, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """dycl_op_conv_maxpool on device tensors: the convolution and the 3x3 /
    stride-2 / pad-1 max-pool after it in one launch; returns the pooled
    y [n, (Ho - 1) // 2 + 1, (Wo - 1) // 2 + 1, cout] bf16."""
    n, H, W, cin = x.shape
    Ho, Wo = (H + 2 * pad - k) // stride + 1, (W + 2 * pad - k) // stride + 1
    Hp, Wp = (Ho - 1) // 2 + 1, (Wo - 1) // 2 + 1
    y = out if out is not None else torch.empty((n, Hp, Wp, cout), dtype=torch.bfloat16, device=x.device)
    s = stream if stream is not None else torch.cuda.current_stream(x.device)
    ptr = lambda t: None if t is None else t.data_ptr()  # noqa: E731
    check(lib.dycl_op_conv_maxpool(x.data_ptr(), n, H, W, cin, packed.data_ptr(), cout, k, stride, pad, ptr(scale),
                                   ptr(shift), act, y.data_ptr(), s.cuda_stream))
    return y


def conv_pair(x: torch.Tensor, packed3: torch.Tensor, scale3: torch.Tensor, shift3: torch.Tensor, res, c3: int,
              packed1: torch.Tensor, scale1: torch.Tensor, shift1: torch.Tensor, c1: int, stream=None):
    """dycl_op_conv_pair on device tensors: x [n, H, W, cin] bf16, the two
    layers' packed 1x1 weights, float32 scale / shift vectors and an optional
    bf16 residual of the first; returns (y3 [n, H, W, c3], y1 [n, H, W, c1])."""
    n, H, W, cin = x.shape
    y3 = torch.empty((n, H, W, c3), dtype=torch.bfloat16, device=x.device)
    y1 = torch.empty((n, H, W, c1), dtype=torch.bfloat16, device=x.device)
    s = stream if stream is not None else torch.cuda.current_stream(x.device)
    check(lib.dycl_op_conv_pair(x.data_ptr(), n, H, W, cin, packed3.data_ptr(), scale3.data_ptr(), shift3.data_ptr(),
                                None if res is None else res.data_ptr(), c3, y3.data_ptr(), packed1.data_ptr(),
                                scale1.data_ptr(), shift1.data_ptr(), c1, y1.data_ptr(), s.cuda_stream))
    return y3, y1


def conv(x: torch.Tensor, packed: torch.Tensor, cout: int, k: int, stride: int, pad: int, scale=None, shift=None,
         res=None, act: int = 0, out: torch.Tensor | None = None, stream=None, workspace="auto") -> torch.Tensor:
    """dycl_op_conv on device tensors: x [n, H, W, cin] bf16, packed weights
    on the device (int16 / uint16 storage), optional float32 scale / shift
    [cout] and bf16 residual; returns y [n, Ho, Wo, cout] bf16.  workspace:
    "auto" allocates what a K-split layer needs (as dycl_run splits), None
    runs it unsplit, or a device tensor."""
    n, H, W, cin = x.shape
    Ho, Wo = (H + 2 * pad - k) // stride + 1, (W + 2 * pad - k) // stride + 1
    y = out if out is not None else torch.empty((n, Ho, Wo, cout), dtype=torch.bfloat16, device=x.device)
    s = stream if stream is not None else torch.cuda.current_stream(x.device)
    ptr = lambda t: None if t is None else t.data_ptr()  # noqa: E731
    if isinstance(workspace, str):
        nb = conv_workspace_bytes(n, H, W, cin, cout, k, stride, pad)
        workspace = torch.empty(nb, dtype=torch.uint8, device=x.device) if nb else None
    wsb = workspace.numel() * workspace.element_size() if workspace is not None else 0
    check(lib.dycl_op_conv(x.data_ptr(), n, H, W, cin, packed.data_ptr(), cout, k, stride, pad, ptr(scale), ptr(shift),
                         ptr(res), act, y.data_ptr(), ptr(workspace), wsb, s.cuda_stream))
    return y
