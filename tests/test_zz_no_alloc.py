"""spexis_accept_noalloc (acceptance in the library's static scratch array, for callers that cannot
allocate) against spexis_accept with a caller-provided workspace: the same outputs bit for bit, on
two calls in a row, the second with a smaller problem, through the C ABI."""
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


def outputs(B, K, seq_lens):
    acc = torch.full((B,), -9, dtype=torch.int32, device="cuda")
    toks = torch.full((B, K + 1), -9, dtype=torch.int32, device="cuda")
    stat = torch.full((B,), -9, dtype=torch.int32, device="cuda")
    sl = torch.as_tensor(seq_lens, device="cuda").clone()
    return acc, toks, stat, sl


def run_both(kind, spec, batch, target, draft, ids, ua, us, temperature):
    K = batch.max_k
    qsl = torch.as_tensor(batch.qsl, device="cuda")
    ref = outputs(batch.B, K, batch.seq_lens)
    ws = torch.empty(sx.spexis_accept_workspace_size(batch.B, spec.vocab, K), dtype=torch.uint8, device="cuda")
    sx.spexis_accept(kind, qsl, target, draft, ids, ua, us, K, ref[0], ref[1], ref[2], ws,
                     temperature=temperature, seq_lens_inout=ref[3])
    got = outputs(batch.B, K, batch.seq_lens)
    sx.spexis_accept_noalloc(kind, qsl, target, draft, ids, ua, us, K, got[0], got[1], got[2],
                             temperature=temperature, seq_lens_inout=got[3])
    torch.cuda.synchronize()
    for r, g in zip(ref, got):
        assert torch.equal(r, g)
    return [t.cpu().numpy() for t in got]


def test_noalloc_accept_equals_workspace_accept_on_two_calls():
    # call 1: the 512-sequence, 152064-entry workload with logits (3.3 MiB of scratch, test rounds)
    spec = wl.WORKLOADS[5]
    batch = wl.make_batch(spec)
    acc = wl.make_accept_inputs(spec, batch, device="cuda")
    say(f"[noalloc] call 1: logits B={batch.B} V={spec.vocab} max_k={batch.max_k} "
        f"workspace={sx.spexis_accept_workspace_size(batch.B, spec.vocab, batch.max_k)}")
    a, t, s, _ = run_both(sx.SPEXIS_INPUT_LOGITS, spec, batch, acc.target_logits, acc.draft_logits, acc.draft_ids,
                          acc.u_accept, acc.u_sample, acc.temperature)
    assert (s == 0).all()
    del acc
    # call 2: a smaller batch (16 sequences of workload 2's shape) with probabilities; the
    # scratch still holds call 1's contents.  Also checked against the oracle.
    spec2 = wl.spec_with(2, batch=16)
    batch2 = wl.make_batch(spec2)
    acc2 = wl.make_accept_inputs(spec2, batch2, device="cuda")
    p = oracle.softmax(acc2.target_logits.cpu().numpy(), acc2.temperature)
    q = oracle.softmax(acc2.draft_logits.cpu().numpy(), acc2.temperature)
    say(f"[noalloc] call 2: probs B={batch2.B} V={spec2.vocab}")
    a2, t2, s2, sl2 = run_both(sx.SPEXIS_INPUT_PROBS, spec2, batch2, torch.as_tensor(p, device="cuda"),
                               torch.as_tensor(q, device="cuda"), acc2.draft_ids, acc2.u_accept, acc2.u_sample, 1.0)
    ra, rt, rs, rsl = oracle.accept(batch2.qsl, p, q, acc2.draft_ids.cpu().numpy(), acc2.u_accept.cpu().numpy(),
                                    acc2.u_sample.cpu().numpy(), max_k=batch2.max_k, seq_lens=batch2.seq_lens)
    np.testing.assert_array_equal(a2, ra)
    np.testing.assert_array_equal(t2, rt)
    np.testing.assert_array_equal(s2, rs)
    np.testing.assert_array_equal(sl2, rsl)
    say(f"[noalloc] both calls equal the workspace entry point (accepted means {a.mean():.3f}, {a2.mean():.3f})")


def test_noalloc_accept_rejects_a_problem_beyond_the_scratch():
    # 512 sequences with up to 32 drafts over 2^18 entries need more than 16 MiB: rejected on the
    # host before any launch, outputs untouched
    B, V, K = 512, 1 << 18, 32
    assert sx.spexis_accept_workspace_size(B, V, K) > sx.SPEXIS_ACCEPT_NOALLOC_SCRATCH_BYTES
    row = torch.zeros((B, V), dtype=torch.float32, device="cuda")
    u = torch.zeros(B, dtype=torch.float32, device="cuda")
    acc, toks, stat, _ = outputs(B, K, np.zeros(B, np.int32))
    with pytest.raises(sx.SpexisError) as e:
        sx.spexis_accept_noalloc(sx.SPEXIS_INPUT_PROBS, torch.arange(B + 1, dtype=torch.int32, device="cuda"), row,
                                 None, None, None, u, K, acc, toks, stat)
    assert e.value.code == sx.SPEXIS_ERR_UNSUPPORTED and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert (acc == -9).all() and (toks == -9).all()
