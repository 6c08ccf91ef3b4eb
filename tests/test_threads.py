"""Calls from several host threads at once, each thread on its own stream with
its own workspaces and outputs: every result is bit-identical to the same call
made alone (the library keeps no state between calls other than what the
caller's workspace holds), and matches the fp64 oracle."""
import threading

import numpy as np
import pytest
import torch

from harness import AttnProblem, check_close

pytestmark = pytest.mark.gpu

N_SINK, WINDOW = 4, 256


def _problems():
    return [AttnProblem(31, 2, 3, 8, 2, 128, [700, 1500, 33]),
            AttnProblem(32, 1, 2, 16, 4, 64, [2000, 90])]


def _calls(prob, stream, reps):
    """`reps` Local + Full calls on `stream`; the results, on the host."""
    P = prob.P
    got = []
    with torch.cuda.stream(stream):
        ws_l = torch.zeros(P.attn_workspace_size(prob.shape, N_SINK, WINDOW), dtype=torch.uint8, device="cuda")
        ws_f = torch.zeros(P.attn_workspace_size(prob.shape, 0, 0), dtype=torch.uint8, device="cuda")
        for _ in range(reps):
            lo, ll = prob.new_out(np.nan)
            fo, fl = prob.new_out(np.nan)
            P.local_decode_attn(prob.shape, prob.inp, N_SINK, WINDOW, lo, ll, ws_l, stream=stream)
            P.full_decode_attn(prob.shape, prob.inp, 0, None, None, None, fo, fl, ws_f, stream=stream)
            got.append((lo, ll, fo, fl))
    stream.synchronize()
    return [tuple(t.cpu() for t in g) for g in got]


def test_concurrent_host_threads_match_single_calls():
    probs = _problems()
    torch.cuda.synchronize()
    alone = [_calls(p, torch.cuda.Stream(), 1)[0] for p in probs]
    for p, (lo, ll, fo, fl) in zip(probs, alone):
        ref_o, ref_l, _ = p.oracle_local(N_SINK, WINDOW)
        check_close(lo.numpy(), ref_o, "local out")
        check_close(ll.numpy(), ref_l, "local lse")
        ref_o, ref_l, _ = p.oracle_full()
        check_close(fo.numpy(), ref_o, "full out")
        check_close(fl.numpy(), ref_l, "full lse")

    jobs = [(i % len(probs), torch.cuda.Stream()) for i in range(4)]
    results, errors = [None] * len(jobs), []

    def work(j):
        try:
            results[j] = _calls(probs[jobs[j][0]], jobs[j][1], 5)
        except BaseException as e:   # surfaced in the main thread
            errors.append(e)

    threads = [threading.Thread(target=work, args=(j,)) for j in range(len(jobs))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=60)
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    if errors:
        raise errors[0]
    for (pi, _), res in zip(jobs, results):
        for rep in res:
            for got, ref in zip(rep, alone[pi]):
                assert torch.equal(got, ref)
