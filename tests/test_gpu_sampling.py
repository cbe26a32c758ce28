"""Deterministic sampling on the GPU (pgsr_sample_tokens) against the oracle
(oracle/sampling.py) on the same seeded logits: the same token wherever the
oracle's best fp32 score beats the second by more than the two sides'
logarithms can disagree; at a closer race, a token whose oracle score is
within that margin of the best.  Greedy rows must match exactly."""
import numpy as np
import pytest
import torch

from oracle import sampling as S
from gpu_helpers import log

from paper_2609_04875_amd import sample_tokens, sample_workspace_bytes

pytestmark = pytest.mark.gpu

# fp32 logs of the two sides may differ by a few ulp; scores stay below ~40
MARGIN = 2e-5


def _logits(rng, n, vocab, dtype):
    x = (rng.standard_normal((n, vocab)) * 3).astype(np.float32)
    t = torch.from_numpy(x).cuda().to(dtype)
    return t, t.float().cpu().numpy().astype(np.float64)


def _check(got, logits64, T, seed, streams, positions):
    want, gaps = S.sample(logits64, T, seed, streams, positions)
    for i, (g, w, gap) in enumerate(zip(got, want, gaps)):
        if g == w:
            continue
        assert T > 0 and gap < MARGIN, f"row {i}: got {g}, want {w}, gap {gap}"
        l = logits64[i].astype(np.float32)
        u = S.uniforms(logits64.shape[1], positions[i], streams[i], seed).astype(np.float32)
        score = l / np.float32(T) - np.log(-np.log(u))
        assert score[g] >= score.max() - MARGIN, f"row {i}: token {g} is not a near-best pick"


@pytest.mark.parametrize("vocab,dtype,split", [(1000, torch.float32, False), (32003, torch.bfloat16, False),
                                               (32003, torch.bfloat16, True), (128256, torch.bfloat16, True)])
@pytest.mark.parametrize("T", [0.0, 0.7])
def test_sampling_matches_oracle(vocab, dtype, split, T):
    log(f"sampling vocab={vocab} {dtype} split={split} T={T}")
    rng = np.random.default_rng(vocab + int(10 * T))
    n = 6
    logits, l64 = _logits(rng, n, vocab, dtype)
    streams = [int(x) for x in rng.integers(0, 1000, size=n)]
    positions = [int(x) for x in rng.integers(0, 100000, size=n)]
    ws = torch.empty(max(sample_workspace_bytes(n, vocab), 1), dtype=torch.uint8, device="cuda") if split else None
    got = sample_tokens(logits, T, 1234, streams, positions, workspace=ws).cpu().numpy()
    _check(got, l64, T, 1234, streams, positions)


def test_many_rows_and_determinism():
    rng = np.random.default_rng(9)
    n, vocab = 150, 5000                       # three launches of up to 64 rows
    logits, l64 = _logits(rng, n, vocab, torch.bfloat16)
    streams = list(range(n))
    positions = [7] * n
    a = sample_tokens(logits, 0.7, 5, streams, positions).cpu().numpy()
    b = sample_tokens(logits, 0.7, 5, streams, positions).cpu().numpy()
    assert (a == b).all()
    _check(a, l64, 0.7, 5, streams, positions)
    c = sample_tokens(logits, 0.7, 6, streams, positions).cpu().numpy()
    assert not (a == c).all()


def test_ties_and_nan():
    x = torch.tensor([[1.0, 3.0, 3.0, float("nan")], [float("nan")] * 4, [-1.0, -0.0, 0.0, -2.0]],
                     device="cuda")
    got = sample_tokens(x, 0.0, 0, [0, 0, 0], [0, 0, 0]).cpu().tolist()
    assert got == [1, 0, 1]


def test_frequencies_follow_softmax():
    """Gumbel-max on the GPU: token frequencies over many positions follow
    softmax(l / T) (a property that holds independently of the oracle)."""
    l = torch.tensor([[0.5, -1.0, 2.0, 0.0, 1.0]], device="cuda").repeat(4000, 1).contiguous()
    T = 0.7
    got = sample_tokens(l, T, 3, [1] * 4000, list(range(4000))).cpu().numpy()
    freq = np.bincount(got, minlength=5) / 4000
    p = np.exp(np.array([0.5, -1.0, 2.0, 0.0, 1.0]) / T)
    p /= p.sum()
    assert np.abs(freq - p).max() < 0.03
