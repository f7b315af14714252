"""Shared helpers of the GPU parity tests: moving storage arrays between the
oracle (numpy bit patterns) and device tensors, bitwise comparison."""
import numpy as np
import torch

TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16, "f8": torch.float8_e4m3fn,
            "u32": torch.int32}
NP_STORAGE = {"f32": np.float32, "bf16": np.uint16, "f16": np.uint16, "f8": np.uint8, "u32": np.uint32}
INT_VIEW = {"f32": torch.int32, "bf16": torch.int16, "f16": torch.int16, "f8": torch.int8, "u32": torch.int32}
NP_INT = {"f32": np.int32, "bf16": np.int16, "f16": np.int16, "f8": np.int8, "u32": np.int32}


def empty(dt, n, device="cuda"):
    return torch.empty(n, dtype=TORCH_DT[dt], device=device)


def to_storage(t, dt):
    """Device tensor -> numpy array of the oracle's storage type (bit patterns)."""
    raw = t.detach().contiguous().view(INT_VIEW[dt]).cpu().numpy()
    return raw.view(NP_STORAGE[dt])


def from_storage(arr, dt, device="cuda"):
    a = np.ascontiguousarray(arr).view(NP_INT[dt])
    return torch.from_numpy(a).to(device).view(TORCH_DT[dt])


def assert_bits_equal(got, ref, what=""):
    g = np.ascontiguousarray(got).view(np.uint8)
    r = np.ascontiguousarray(ref).view(np.uint8)
    assert g.shape == r.shape, (what, g.shape, r.shape)
    if not np.array_equal(g, r):
        isz = np.ascontiguousarray(ref).itemsize
        bad = np.nonzero((g.reshape(-1, isz) != r.reshape(-1, isz)).any(axis=1))[0]
        raise AssertionError("%s: %d elements differ, first at %s: got %s ref %s" % (
            what, bad.size, bad[:5], np.ascontiguousarray(got).ravel()[bad[:5]],
            np.ascontiguousarray(ref).ravel()[bad[:5]]))


def same_result(gpu, ref):
    """Check records equal field by field (floats bitwise as fp32)."""
    g = gpu.as_dict() if hasattr(gpu, "as_dict") else dict(gpu)
    for k in ("n", "mismatches", "nan_count", "argmax_abs"):
        assert int(g[k]) == int(ref[k]), (k, g[k], ref[k])
    for k in ("max_abs", "max_rel"):
        a = np.float32(g[k]).view(np.uint32)
        b = np.float32(ref[k]).view(np.uint32)
        assert a == b, (k, g[k], ref[k])
