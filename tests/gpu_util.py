"""Helpers shared by the GPU tests: upload seeded host arrays, compare with the
oracle under the stated tolerance, and run the library entry points."""
import math
import sys

import numpy as np
import torch

ATOL, RTOL, RMS_GATE = 2e-2, 1e-2, 5e-3


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def bf16_dev(a: np.ndarray) -> torch.Tensor:
    """uint16 bf16 bit patterns -> device bf16 tensor (same bits)."""
    t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16))
    return t.cuda().view(torch.bfloat16)


def i32_dev(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def host_bits(t: torch.Tensor) -> np.ndarray:
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def assert_attn_close(gpu: torch.Tensor, ref: np.ndarray, what: str):
    """Elementwise |gpu - ref| <= ATOL + RTOL*|ref| and RMS-relative error <= RMS_GATE."""
    g = gpu.float().cpu().numpy().astype(np.float64).reshape(ref.shape)
    assert np.isfinite(g).all(), "%s: non-finite GPU output" % what
    err = np.abs(g - ref)
    tol = ATOL + RTOL * np.abs(ref)
    rms = math.sqrt(float(np.mean((g - ref) ** 2)))
    rms_ref = math.sqrt(float(np.mean(ref ** 2))) or 1.0
    log("%s: max|err| %.3e  max rel %.3e  rms-rel %.3e  (%d values)" % (
        what, err.max(), (err / np.maximum(np.abs(ref), 1e-6)).max(), rms / rms_ref, ref.size))
    bad = err > tol
    assert not bad.any(), "%s: %d of %d values outside tolerance, worst err %.3e at %s" % (
        what, int(bad.sum()), ref.size, err.max(), np.unravel_index(np.argmax(err - tol), err.shape))
    assert rms / rms_ref <= RMS_GATE, "%s: rms-relative error %.3e > %.1e" % (what, rms / rms_ref,
                                                                              RMS_GATE)


class DevicePool:
    """A pool uploaded to the GPU and wrapped by kv_pool_create, with an optional
    device ring (whole all-layer blocks) for host-staged copies."""

    def __init__(self, kv_mod, pool_host: np.ndarray, head_dim: int, ring_blocks: int = 0):
        nl, nb, _, hkv, _ = pool_host.shape
        self.kv_mod = kv_mod
        self.data = bf16_dev(pool_host)
        self.ring = None
        if ring_blocks:
            per_block = nl * 2 * hkv * 16 * head_dim * 2
            self.ring = torch.empty(ring_blocks * per_block, dtype=torch.uint8, device="cuda")
        self.pool = kv_mod.kv_pool_create(self.data, nl, nb, hkv, head_dim, 16)
        self.shape = pool_host.shape

    def host(self) -> np.ndarray:
        torch.cuda.synchronize()
        return host_bits(self.data).reshape(self.shape)


def run_decode(kv_mod, dp: DevicePool, q, tables, lens, scale, k_new=None, v_new=None,
               layer=0, workspace=None):
    s, hq, d = q.shape
    out = torch.empty((s, hq, d), dtype=torch.bfloat16, device="cuda")
    if workspace is None:
        nbytes = kv_mod.decode_workspace_bytes(dp.pool, s, hq, tables.shape[1])
        workspace = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    kv_mod.paged_attn_decode(dp.pool, layer, q, tables, lens, scale, out, workspace, k_new, v_new)
    return out, workspace


def cu_masked_stream(lo: int, hi: int):
    """A torch stream whose kernels may run only on CUs lo .. hi-1 (through
    hipExtStreamCreateWithCUMask of the runtime this process loaded), or None
    when that runtime entry is unavailable.  Returns (stream, handle)."""
    import ctypes
    import os
    lib = None
    for line in open("/proc/self/maps"):
        parts = line.split()
        if len(parts) >= 6 and "libamdhip64" in os.path.basename(parts[-1]):
            lib = ctypes.CDLL(parts[-1])
            break
    if lib is None or not hasattr(lib, "hipExtStreamCreateWithCUMask"):
        return None
    mask = (ctypes.c_uint32 * 32)()
    for cu in range(lo, hi):
        mask[cu // 32] |= 1 << (cu % 32)
    h = ctypes.c_void_p()
    if lib.hipExtStreamCreateWithCUMask(ctypes.byref(h), 32, mask) != 0:
        return None
    return torch.cuda.ExternalStream(h.value), (lib, h)


def destroy_stream(handle):
    lib, h = handle
    lib.hipStreamDestroy(h)


def key_ramp(shape: str, nblk: int, j: np.ndarray) -> np.ndarray:
    """Per-block K scale for block positions j of an nblk-block context.

    rising: 1 -> 10 along the context, so the running max is raised many times;
    spike: 16 on the second-to-last block only, one large late raise;
    falling: 10 -> 1, the first blocks hold the max and nothing is raised.
    """
    t = j / max(nblk - 1, 1)
    if shape == "rising":
        return 1.0 + 9.0 * t
    if shape == "falling":
        return 10.0 - 9.0 * t
    if shape == "spike":
        return np.where(j == max(nblk - 2, 0), 16.0, 1.0)
    raise ValueError(shape)


def scale_keys(pool: np.ndarray, tables: np.ndarray, ctx_tokens, shape: str):
    """Multiply the K tiles of each session's context blocks by key_ramp (in place,
    rounded to bf16; NaN slots stay NaN).  ``ctx_tokens[s]`` tokens are in the pool."""
    from paper_2606_22983_amd import workloads as W
    for s in range(tables.shape[0]):
        nblk = (int(ctx_tokens[s]) + 15) // 16
        if nblk == 0:
            continue
        j = np.arange(nblk)
        f = key_ramp(shape, nblk, j).astype(np.float32)
        ids = tables[s, :nblk]
        k = W.from_bf16(pool[0, ids, 0])
        pool[0, ids, 0] = W.to_bf16(k * f[:, None, None])

