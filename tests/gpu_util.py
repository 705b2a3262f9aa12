"""Helpers shared by the GPU parity tests (host <-> device, error metrics)."""
import numpy as np

import forge_inputs as fi


def rel_fro(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))


def dev_bf16(bits, device="cuda"):
    from paper_2609_13645_amd import runtime
    return runtime.to_device_bf16(bits, device)


def host_f64(t):
    """bf16 or fp32 device tensor -> fp64 numpy."""
    import torch
    from paper_2609_13645_amd import runtime
    if t.dtype == torch.bfloat16:
        return fi.bf16_bits_to_f64(runtime.to_host_bits(t))
    return t.detach().cpu().numpy().astype(np.float64)


def banner(msg):
    print(f"[gpu-test] {msg}", flush=True)
