"""GPU parity of DGAP's logit-side step (dgap_restore, through the C ABI)
against the fp64 oracle (oracle/dgap.py) on the same seeded rows and weights.

- the window (TopK indices, in order): identical, ties included;
- features: within 1e-5 relative (1e-6 absolute) of the oracle;
- risk r: within 1e-5; the corrected / bypassed decision equal wherever the
  oracle's r is more than 1e-4 away from tau;
- logits: every entry outside a corrected window bit-identical to the
  input; window entries and Delta within 1e-4 of the oracle;
- bitwise reproducible.
"""
import numpy as np
import pytest

from oracle import dgap as odgap
from dgap_inputs import VOCAB, gen_logits, gen_weights
from helpers import log

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _run(z, k, w, tau=odgap.TAU):
    from paper_2607_16248_amd import kvq
    dev = torch.device("cuda:0")
    B, V = z.shape
    t = {n: torch.from_numpy(np.ascontiguousarray(getattr(w, n))).to(dev) for n in ("w1", "b1", "w2", "c1", "cb1", "c2")}
    p = kvq.dgap_params(V, k, tau, t["w1"], t["b1"], t["w2"], w.b2, t["c1"], t["cb1"], t["c2"], w.cb2)
    logits = torch.from_numpy(z.copy()).to(dev)
    ws = torch.empty(kvq.dgap_workspace_bytes(B, V, k), dtype=torch.uint8, device=dev)
    info = torch.full((B, kvq.dgap_info_floats(k)), float("nan"), dtype=torch.float32, device=dev)
    kvq.dgap_restore(p, logits, B, ws, info=info)
    torch.cuda.synchronize()
    return logits.cpu().numpy(), info.cpu().numpy()


def _check_row(z, out, info, k, w, tau=odgap.TAU):
    ref = odgap.restore(z, k, w, tau)
    idx = info[16:16 + k].view(np.int32)
    assert np.array_equal(idx, ref.idx), (idx[:8], ref.idx[:8])
    phi = info[4:16].astype(np.float64)
    err = np.abs(phi - ref.phi) / np.maximum(np.abs(ref.phi), 0.1)
    assert err.max() <= 1e-5, (np.argmax(err), phi, ref.phi)
    assert abs(info[0] - ref.risk) <= 1e-5, (info[0], ref.risk)
    decided = info[1] == 1.0
    if abs(ref.risk - tau) > 1e-4:
        assert decided == ref.corrected
    outside = np.ones(z.size, bool)
    if decided:
        outside[idx] = False
        delta = info[16 + k:16 + 2 * k].astype(np.float64)
        want = odgap.corrector(odgap.candidate_features(z, k), ref.phi, w)
        assert np.abs(delta - want).max() <= 1e-4
        assert np.abs(out[idx].astype(np.float64) - (z[idx].astype(np.float64) + want)).max() <= 1e-4
    else:
        assert np.all(info[16 + k:16 + 2 * k] == 0)
    assert np.array_equal(out[outside].view(np.uint32), z[outside].view(np.uint32))
    return ref, decided


CASES = [
    ("llama3_8b", 128, "peaked", 20.0),
    ("qwen2_5_14b", 128, "peaked", 20.0),
    ("qwen2_5_14b", 64, "flat", 0.0),
    ("mistral_7b", 32, "peaked", -20.0),
    ("mistral_7b", 16, "ties", 20.0),
    ("llama3_8b", 256, "ties", 20.0),
]


@pytest.mark.parametrize("model,k,kind,bias", CASES, ids=[f"{m}_k{k}_{kd}_{b:+.0f}" for m, k, kd, b in CASES])
def test_restore_matches_oracle(model, k, kind, bias):
    V = VOCAB[model]
    z = gen_logits(V, batch=2, seed=k, kind=kind)
    w = gen_weights(seed=k, det_bias=bias)
    out, info = _run(z, k, w)
    for b in range(2):
        ref, dec = _check_row(z[b], out[b], info[b], k, w)
        log(f"[dgap] {model} k={k} {kind} row {b}: r={info[b][0]:.6f} (oracle {ref.risk:.6f}) corrected={dec}")


def test_random_detector_over_many_rows():
    # a batch of 16 rows with the random detector: some rows corrected, some not
    V, k = VOCAB["qwen2_5_14b"], 128
    z = gen_logits(V, batch=16, seed=99, kind="flat")
    z[::2] = gen_logits(V, batch=8, seed=98, kind="peaked")
    w = gen_weights(seed=5, det_bias=0.0, scale=3.0)
    out, info = _run(z, k, w)
    decisions = [_check_row(z[b], out[b], info[b], k, w)[1] for b in range(16)]
    log(f"[dgap] random detector: {sum(decisions)} of 16 rows corrected")


@pytest.mark.parametrize("V,k", [(16, 16), (300, 256), (2048, 256), (2049, 8), (6144, 100)])
def test_edge_shapes(V, k):
    # whole vocabulary as the window, chunks shorter than the window, one
    # logit past a chunk edge, a window size that is not a power of two
    z = gen_logits(max(V, 32), batch=1, seed=V)[:, :V].copy()
    w = gen_weights(seed=1, det_bias=20.0)
    out, info = _run(z, k, w)
    _check_row(z[0], out[0], info[0], k, w)


def test_exact_ties_at_the_window_edge():
    # 4000 equal logits below 10 distinct leaders: the window takes the
    # lowest indices among the equal ones
    V, k = 8192, 32
    z = np.zeros((1, V), np.float32)
    z[0, 4000:] = -1.0
    lead = np.random.default_rng(0).choice(V, 10, replace=False)
    z[0, lead] = np.arange(10, 0, -1, dtype=np.float32) + 5.0
    w = gen_weights(seed=2, det_bias=20.0)
    out, info = _run(z, k, w)
    _check_row(z[0], out[0], info[0], k, w)


def test_bitwise_reproducible():
    V, k = VOCAB["llama3_8b"], 128
    z = gen_logits(V, batch=4, seed=3)
    w = gen_weights(seed=3, det_bias=20.0)
    a, ia = _run(z, k, w)
    b, ib = _run(z, k, w)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert np.array_equal(ia.view(np.uint32), ib.view(np.uint32))
