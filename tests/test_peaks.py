"""The peak-rate microbenchmarks (libcppeaks.so): exported symbols on the CPU;
on the GPU, the streaming read's result against a host emulation of its
access pattern, and a sane MFMA-loop run."""

import os
import re

import numpy as np
import pytest

from paper_2606_09061_amd import peaks

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_function():
    src = open(os.path.join(ROOT, "include", "cp_peaks.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = sorted(set(re.findall(r"\b(cpk_[a-z_]+)\s*\(", src)))
    assert names == sorted(peaks.exported_symbols())
    lib = peaks.load()
    for n in names:
        assert hasattr(lib, n)


def _read_stream_host(words, blocks):
    """words: uint32 [n16, 4]; the kernel's grid-stride XOR per thread."""
    n = len(words)
    S = blocks * 256
    out = np.zeros(S, np.uint32)
    for t in range(S):
        x = np.uint32(0)
        i = t
        while i + 3 * S < n:
            x ^= words[i, 0] ^ words[i + S, 1] ^ words[i + 2 * S, 2] ^ words[i + 3 * S, 3]
            i += 4 * S
        while i < n:
            x ^= words[i, 0] ^ words[i, 3]
            i += S
        out[t] = x
    return out


@pytest.mark.gpu
def test_read_stream_matches_host_emulation():
    import torch
    dev = torch.device("cuda", 0)
    rng = np.random.default_rng(0)
    for n16, blocks in ((5000, 2), (1 << 14, 4), (7, 1)):
        print(f"read_stream n16={n16} blocks={blocks}", flush=True)
        words = rng.integers(0, 2 ** 32, (n16, 4), dtype=np.uint64).astype(np.uint32)
        src = torch.from_numpy(words.view(np.int32).copy()).to(dev)
        out = torch.empty(blocks * 256, dtype=torch.int32, device=dev)
        peaks.read_stream(src, out, blocks, torch.cuda.current_stream(dev))
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy().view(np.uint32), _read_stream_host(words, blocks))


@pytest.mark.gpu
def test_mfma_loop_runs_and_device_info_is_sane():
    import torch
    dev = torch.device("cuda", 0)
    info = peaks.device_info(0)
    assert info["compute_units"] > 0 and info["clock_khz"] > 0
    ops = torch.randn(4096, device=dev).to(torch.bfloat16)
    out = torch.empty(8 * 256, dtype=torch.float32, device=dev)
    for rnd in (0, 1):
        peaks.mfma_loop(ops, out, 8, 256, 10, rnd, torch.cuda.current_stream(dev))
    torch.cuda.synchronize()
    assert torch.isfinite(out).all()
    with pytest.raises(ValueError):
        peaks.mfma_loop(ops, out, 16, 256, 10, 1, torch.cuda.current_stream(dev))
    assert peaks.load().cpk_mfma_loop(ops.data_ptr(), 512, out.data_ptr(), 8, 96, 10, 1, None) == -1
