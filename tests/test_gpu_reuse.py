"""The warm-up reuse sequence (Sec. 3.3) against the oracle, step by step.

A short drifting sequence runs through the benchmark's reuse driver on a
reduced 480p grid (5 x 30 x 52 = 7,800 tokens, a ragged last block), with the
entropies shifted so that the masks keep about 30 % of the blocks.  After every
step the test checks, on the host:

* refresh step: the fused pass's dense output (Eq. 2) and entropy (Eq. 1) of
  that step's own q, k; the Alg. 1 mask of that step's radii, bit for bit;
* reuse step: the cached mask and lists are the last refresh's, unchanged; the
  output is block-sparse attention (Eq. 16) of that step's q, k, v under the
  cached mask; the fresh mask built for the drift statistic is Alg. 1 of that
  step's radii;
* the drift statistics the driver reports equal the host's count.
"""
import numpy as np
import pytest

import oracle as O
import synth
from _pipeline import (TOL_H_ABS, TOL_H_REL, TOL_O_BF16, OracleTables, log, sample_blocks,
                       to_np_f64)

pytestmark = pytest.mark.gpu


def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


W = synth.workload("reuse_480p").replace(name="reuse_small", heads=2, frames=5)


def _check_lists(mask, cnt, cols):
    NB = mask.shape[-1]
    m2, c2, n2 = mask.reshape(-1, NB), cols.reshape(-1, NB), cnt.reshape(-1)
    assert np.array_equal(n2, m2.sum(axis=1))
    for r in range(m2.shape[0]):
        assert np.array_equal(c2[r, :n2[r]], np.nonzero(m2[r])[0])
        assert (c2[r, n2[r]:] == -1).all()


def test_reuse_sequence_steps_match_oracle():
    _gpu()
    import bench
    import torch
    import paper_2608_02504_amd as tra
    w = W
    tabs = OracleTables(w)
    N, b, NB = w.n_tokens, w.block, w.n_blocks
    assert N % b != 0                                   # ragged last block
    blocks = sample_blocks(w, 4, seed=11)
    all_blocks = list(range(NB))
    seen = {"refresh": 0, "reuse": 0}
    cached = {}
    host_drift = []
    q0 = {}

    def mask_ref(rad, h):
        return O.block_mask_rows(rad[0, h], tabs.perm, b, tabs.F, tabs.H, tabs.W, w.gamma, all_blocks)

    def on_step(t, kind, st):
        seen[kind] += 1
        q, k, v = (to_np_f64(st[n]) for n in ("q", "k", "v"))
        o = to_np_f64(st["o"])
        mask = st["mask"].cpu().numpy().astype(bool)
        cnt, cols = st["cnt"].cpu().numpy(), st["cols"].cpu().numpy()
        rad = st["rad"].cpu().numpy()
        if t == 0:
            q0["q"] = q
        elif t == 1:
            assert not np.array_equal(q, q0["q"]), "q does not drift between steps"
        err = 0.0
        if kind == "refresh":
            H = st["H"].double().cpu().numpy() + st["shift"]
            for h in range(w.heads):
                rows = np.concatenate([tabs.perm[u * b:min((u + 1) * b, N)] for u in blocks[(0, h)]])
                p = O.softmax_rows(O.scores(q[0, h][rows], k[0, h]))
                H_ref = O.entropy_from_probs(p)
                O_ref = (p @ torch.as_tensor(v[0, h])).numpy()
                dH = np.abs(H[0, h][rows] - H_ref)
                assert (dH <= np.maximum(TOL_H_REL * np.abs(H_ref), TOL_H_ABS) + 1e-6 * st["shift"]).all(), \
                    f"step {t} head {h}: entropy max |dH| {dH.max():.3e}"
                err = max(err, float(np.abs(o[0, h][rows] - O_ref).max()))
                assert np.array_equal(mask[0, h], mask_ref(rad, h)), f"step {t} head {h}: refresh mask"
            _check_lists(mask, cnt, cols)
            cached.update(mask=mask, cnt=cnt, cols=cols)
        else:
            assert np.array_equal(mask, cached["mask"]), f"step {t}: cached mask changed"
            assert np.array_equal(cnt, cached["cnt"]) and np.array_equal(cols, cached["cols"]), \
                f"step {t}: cached lists changed"
            fmask = st["fmask"].cpu().numpy().astype(bool)
            for h in range(w.heads):
                sel = list(blocks[(0, h)])
                rows, O_ref = O.masked_attention_rows(q[0, h], k[0, h], v[0, h], tabs.perm, b, sel,
                                                      cached["mask"][0, h][sel])
                err = max(err, float(np.abs(o[0, h][rows] - O_ref).max()))
                assert np.array_equal(fmask[0, h], mask_ref(rad, h)), f"step {t} head {h}: fresh mask"
            host_drift.append(float((cached["mask"] ^ fmask).mean()))
        assert err <= TOL_O_BF16, f"step {t} ({kind}): output max-abs {err:.3e}"
        log(f"step {t} {kind}: output max-abs {err:.3e}, kept {mask.mean():.3f} of the blocks")

    res = bench.reuse_driver(tra, w, steps=7, refresh=5, target_rho=0.3, on_step=on_step)
    assert seen == {"refresh": 2, "reuse": 5}
    assert res["entropy_shift_nats"] > 0
    assert 0.05 < res["retained_fraction_last_mask"] < 0.9, res["retained_fraction_last_mask"]
    assert max(host_drift) > 0                          # the fresh masks do differ from the cached ones
    assert res["mask_drift_hamming_mean"] == pytest.approx(np.mean(host_drift), rel=1e-6, abs=1e-9)
    assert res["mask_drift_hamming_max"] == pytest.approx(np.max(host_drift), rel=1e-6, abs=1e-9)
    assert res["refresh_step_ms"] > 0 and res["reuse_step_ms"] > 0
    log(f"reuse sequence: {res}")
