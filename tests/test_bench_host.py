"""Host-side pieces of the benchmark that its reported numbers rest on,
checked on the CPU: the executed-FLOP count of a block mask (4 d per valid
query-key pair of every kept block pair) against a brute-force count over
token pairs, and the refusal of more than one GPU."""
import subprocess
import sys
from pathlib import Path

import numpy as np

ROOT = Path(__file__).resolve().parents[1]
sys.path.insert(0, str(ROOT))
import bench  # noqa: E402


def test_executed_flops_matches_pair_count():
    rng = np.random.default_rng(3)
    for N, b, d in ((1000, 128, 128), (256, 64, 64), (128, 128, 64)):
        nb = -(-N // b)
        mask = rng.random((2, 3, nb, nb)) < 0.4
        blk = np.arange(N) // b
        pairs = sum(int(mask[i, j][blk][:, blk].sum()) for i in range(2) for j in range(3))
        assert bench.executed_flops(mask, N, b, d) == 4.0 * d * pairs


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, str(ROOT / "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr


def test_kept_fraction_matches_executed_flops():
    """The device-side count the benchmark uses (run here on CPU tensors) equals
    the host count, and its fraction is over 4 d N^2 per (batch, head)."""
    import torch
    rng = np.random.default_rng(4)
    for N, b, d in ((1000, 128, 128), (75600, 128, 128)):
        nb = -(-N // b)
        mask = rng.random((1, 2, nb, nb)) < 0.3
        rho, fl = bench.kept_fraction(torch.from_numpy(mask.astype(np.uint8)), N, b, d)
        assert fl == bench.executed_flops(mask, N, b, d)
        assert abs(rho - fl / (4.0 * d * N * N * 2)) < 1e-15


def test_mask_source_adjusts_entropies():
    """own leaves H alone, entropy subtracts its constant, uniform overwrites H."""
    import torch
    H = torch.tensor([1.0, 2.5, 7.0])
    assert torch.equal(bench.MaskSource("own").apply(H.clone()), H)
    assert torch.equal(bench.MaskSource("entropy", 1.5).apply(H.clone()), H - 1.5)
    assert torch.equal(bench.MaskSource("uniform", 3.0).apply(H.clone()), torch.full_like(H, 3.0))
