"""GPU parity of selective speculation (spexis_select_drafts) against the oracle.

Integer outputs from fp32 scores that both sides form the same way (an fp32 product in draft
order) and order the same way: the bar is bit-exact kept counts, reduced query_start_loc and
keep flags.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2609_34370_amd import spexis as sx
from paper_2609_34370_amd import workloads as wl

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def batch(k):
    return np.concatenate([[0], np.cumsum(np.asarray(k) + 1)]).astype(np.int32)


def gpu_select(qsl, conf, alpha):
    B = len(qsl) - 1
    N = int(qsl[-1]) - B
    kept_k = torch.empty(B, dtype=torch.int32, device="cuda")
    kept_qsl = torch.empty(B + 1, dtype=torch.int32, device="cuda")
    keep = torch.empty(max(N, 1), dtype=torch.int32, device="cuda")
    sx.spexis_select_drafts(torch.as_tensor(qsl, device="cuda"), torch.as_tensor(conf, device="cuda"), alpha,
                            kept_k, kept_qsl, keep[:N])
    torch.cuda.synchronize()
    return kept_k.cpu().numpy(), kept_qsl.cpu().numpy(), keep[:N].cpu().numpy()


def check(qsl, conf, alpha):
    g = gpu_select(qsl, conf, alpha)
    r = oracle.select_drafts(qsl, conf, alpha)
    for a, b in zip(g, r):
        np.testing.assert_array_equal(a, b)
    return g


@pytest.mark.parametrize("B,kmax,alpha", [(1, 4, 0.3), (7, 8, 0.0), (64, 4, 0.15), (512, 8, 0.3), (300, 16, 0.5),
                                          (1000, 3, 0.99)])
def test_select_matches_oracle(B, kmax, alpha):
    rng = np.random.default_rng(B * 31 + kmax)
    k = rng.integers(0, kmax + 1, B)
    conf = rng.random(int(k.sum()), dtype=np.float32)
    kept_k, _, keep = check(batch(k), conf, alpha)
    say(f"[select] B={B} N={int(k.sum())} alpha={alpha}: kept {int(keep.sum())} drafts")


def test_select_ties_and_odd_values():
    rng = np.random.default_rng(5)
    k = rng.integers(0, 9, 200)
    N = int(k.sum())
    conf = np.ones(N, np.float32)                          # all scores tie: the index decides
    check(batch(k), conf, 0.3)
    conf = rng.choice(np.array([0.0, 0.5, 1.0, 2.0, -1.0, np.nan], np.float32), N)   # clamped, many ties
    check(batch(k), conf, 0.25)
    conf = np.full(N, 1e-20, np.float32)                   # prefix products go subnormal, then 0
    check(batch(k), conf, 0.6)
    conf = np.where(rng.random(N) < 0.5, np.float32(-0.0), np.float32(0.75)).astype(np.float32)   # -0 is 0
    check(batch(k), conf, 0.4)
    conf = rng.random(N, dtype=np.float32)                 # one kept draft: rank R = 1
    check(batch(k), conf, float(np.nextafter(np.float32(1.0), np.float32(0.0))))


def test_select_largest_batch():
    rng = np.random.default_rng(6)
    k = np.full(1024, 16)                                  # 16384 drafts, the supported maximum
    conf = rng.uniform(0.5, 1.0, int(k.sum())).astype(np.float32)
    check(batch(k), conf, 0.2)
    # scores are powers of two: large ties split at the threshold across every 1024-draft row
    conf = rng.choice(np.array([1.0, 0.5], np.float32), int(k.sum()))
    for alpha in (0.1, 0.5, 0.9):
        check(batch(k), conf, alpha)


def test_select_on_workload_confidences():
    # confidences q_i(x_i) of the ragged-selective workload's drafts (B=128, k in 0..8,
    # vocabulary 32000; host softmax in fp64)
    spec = wl.WORKLOADS[4]
    b = wl.make_batch(spec)
    acc = wl.make_accept_inputs(spec, b, device="cpu")
    dl = acc.draft_logits.numpy().astype(np.float64) / acc.temperature
    ids = acc.draft_ids.numpy()
    m = dl.max(axis=1, keepdims=True)
    q = np.exp(dl - m)
    conf = (q[np.arange(len(ids)), ids] / q.sum(axis=1)).astype(np.float32)
    for alpha in (0.15, 0.3):
        kept_k, kept_qsl, keep = check(b.qsl, conf, alpha)
        say(f"[select] ragged-selective B=128 alpha={alpha}: kept {int(keep.sum())} of {len(conf)} drafts, "
            f"{int((kept_k == 0).sum())} sequences without drafts")


def test_select_rejects_bad_arguments():
    qsl = torch.as_tensor(batch([2, 3]), device="cuda")
    conf = torch.ones(5, device="cuda")
    out = [torch.empty(2, dtype=torch.int32, device="cuda"), torch.empty(3, dtype=torch.int32, device="cuda"),
           torch.empty(5, dtype=torch.int32, device="cuda")]
    for alpha in (1.0, -0.1, float("nan")):
        with pytest.raises(sx.SpexisError) as e:
            sx.spexis_select_drafts(qsl, conf, alpha, *out)
        assert e.value.code == sx.SPEXIS_ERR_INVALID_ARGUMENT
    big = torch.as_tensor(batch([16385]), device="cuda")
    with pytest.raises(sx.SpexisError) as e:
        sx.spexis_select_drafts(big, torch.ones(16385, device="cuda"), 0.2, out[0][:1], out[1][:2],
                                torch.empty(16385, dtype=torch.int32, device="cuda"))
    assert e.value.code == sx.SPEXIS_ERR_UNSUPPORTED
