"""Helpers shared by the GPU tests: run a synthetic model through the C ABI and compare."""
import json
import os
import sys

import numpy as np

import synth
from oracle import forward as oracle_forward


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def torch_dev():
    import torch
    return torch, torch.device("cuda", 0)


def to_device(x: np.ndarray):
    torch, dev = torch_dev()
    if x.dtype == np.uint16:
        x = x.view(np.int16)
    return torch.from_numpy(np.ascontiguousarray(x)).to(dev)


def out_shape(model, batch):
    if model.arch == "mlp":
        return (batch, model.dims["width"])
    if model.arch == "resnet50":
        return (batch, model.dims["classes"])
    return (batch, model.dims["seq"], model.dims["d"])


def make_runtime(models, batch_max=1, arena_bytes=None, **kw):
    import paper_2306_03622_amd as tp
    descs = [tp.ModelDesc.of(m) for m in models]
    ws = max(tp.tp_workspace_bytes(d, batch_max) for d in descs)
    if arena_bytes is None:
        arena_bytes = sum(m.total_bytes for m in models) + (1 << 20)
    kw.setdefault("direct_max_bytes", 0)        # cold requests take the swap path unless a test asks
    rt = tp.Runtime(arena_bytes, ws, **kw)
    ids = [rt.register(d, m.blob()) for d, m in zip(descs, models)]
    return rt, ids


def infer(rt, mid, model, x_np, stream=None):
    """One request; returns the fp32 output on the host."""
    torch, dev = torch_dev()
    x = to_device(x_np)
    out = torch.full(out_shape(model, x_np.shape[0]), float("nan"), dtype=torch.float32, device=dev)
    s = stream or torch.cuda.Stream(device=dev)
    torch.cuda.synchronize()
    rt.infer(mid, x, out, stream=s)
    s.synchronize()
    return out.cpu().numpy()


# where GPU tests leave their records: $TP_RESULTS_DIR, else results/ at the repository root
RESULTS_DIR = os.environ.get("TP_RESULTS_DIR") or os.path.join(
    os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "results")
# every parity check appends its achieved error here (one JSON object per line), so a GPU
# run leaves a record of the errors behind its pass/fail verdicts
PARITY_LOG = os.environ.get("TP_PARITY_LOG", os.path.join(RESULTS_DIR, "parity_errors.jsonl"))


def record_parity(model, batch, err, tol):
    rec = {"test": os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0], "arch": model.arch,
           "dtype": model.dtype, "dims": {k: v for k, v in model.dims.items() if isinstance(v, (int, str))},
           "batch": int(batch), "max_normwise_error": float(err), "tol": tol}
    try:
        os.makedirs(os.path.dirname(PARITY_LOG), exist_ok=True)
        with open(PARITY_LOG, "a") as f:
            f.write(json.dumps(rec) + "\n")
    except OSError as e:          # a read-only tree must not fail the check itself
        log(f"  (parity record not written: {e})")


def check_parity(got, model, x_np, tol):
    ref = oracle_forward.forward(model, x_np)
    err = oracle_forward.normwise_error(got, ref)
    log(f"  normwise error per sample: max {err.max():.3e} (tol {tol})")
    assert np.all(np.isfinite(got)), "non-finite output"
    record_parity(model, x_np.shape[0], err.max(), tol)
    assert err.max() <= tol, (err.max(), tol)
    return err


def pack_rows16x128(w: np.ndarray) -> np.ndarray:
    """Blocked order of a bf16 [N][K] matrix used for skinny-batch MLP weights: blocks of 16
    rows x 128 columns, each ordered [32-column group][8-column slot][row][8 elements]."""
    n, k = w.shape
    return w.reshape(n // 16, 16, k // 128, 4, 4, 8).transpose(0, 2, 3, 4, 1, 5).reshape(-1)


def expected_host_image(model) -> np.ndarray:
    """The library's pinned host image of `model` (bf16 MLPs with width % 128 == 0 are blocked)."""
    img = model.blob().copy()
    if model.arch == "mlp" and model.dtype == "bf16" and model.dims["width"] % 128 == 0:
        for t in model.tensors:
            if t.role == "w":
                w = img[t.offset:t.offset + t.nbytes].view(np.uint16).reshape(t.shape)
                img[t.offset:t.offset + t.nbytes] = pack_rows16x128(w).view(np.uint8)
    return img
