"""Shared helpers for the GPU parity tests: device upload and comparison."""
import numpy as np

import oracle

TOL = {"fp32": 1e-4, "bf16": 2e-2}


def torch_dtype(name):
    import torch
    return torch.bfloat16 if name == "bf16" else torch.float32


def dev(a, dtype: str):
    """Numpy array (bf16-representable when dtype is bf16) -> contiguous cuda tensor."""
    import torch
    if a is None:
        return None
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda").to(torch_dtype(dtype)).contiguous()


def dev_weights(w, dtype: str):
    out = {}
    for key, val in w.items():
        if isinstance(val, list):
            out[key] = [(dev(a, dtype), dev(b, dtype)) for a, b in val]
        elif isinstance(val, tuple):
            out[key] = (dev(val[0], dtype), dev(val[1], dtype))
        else:
            out[key] = dev(val, dtype)
    return out


def host(t):
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def assert_close(got, ref, dtype: str, what: str):
    err = oracle.max_rel_err(got, ref)
    tol = TOL[dtype]
    print(f"  {what}: max rel err {err:.3e} (tol {tol:g})", flush=True)
    assert err <= tol, f"{what}: max relative error {err:.3e} > {tol:g}"
    return err
