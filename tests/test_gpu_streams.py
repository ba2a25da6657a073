"""Calls on separate streams and from separate host threads.

Each call only enqueues work on the stream it is given and keeps no state between
calls, so two rounds with their own buffers and workspaces may run at the same time:
on two non-default streams from one thread, and from two host threads, the outputs must
equal those of the same rounds run one after the other, bit for bit.
"""
import threading

import numpy as np
import pytest

from gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2607_25852_amd import binding
    binding.load()
    return torch


OUTS = ("qo", "keep", "attn_out", "attn_lse", "accept_len", "out_tokens", "flags")


def _snapshot(rnd):
    return {k: getattr(rnd, k).clone() for k in OUTS}


def _poison(rnd):
    for k in OUTS:
        t = getattr(rnd, k)
        if t.dtype.is_floating_point:
            t.fill_(-3.0)
        else:
            t.fill_(-7)


def _same(a, b):
    for k in OUTS:
        assert a[k].shape == b[k].shape and bool((a[k] == b[k]).all()), k


def test_two_streams_and_two_threads(dev):
    torch = dev
    from paper_2607_25852_amd import synth
    from paper_2607_25852_amd.round import DeviceRound
    say("streams: c16_b16 and sweep_mtp_c8 rounds")
    rounds = [DeviceRound(synth.CONFIGS["c16_b16"], kind="logits"),
              DeviceRound(synth.CONFIGS["sweep_mtp_c8"], kind="logits")]
    refs = []
    for r in rounds:
        _poison(r)
        r.run()
        torch.cuda.synchronize()
        refs.append(_snapshot(r))
    # two non-default streams, launched from one thread, several times over
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for rep in range(3):
        for r in rounds:
            _poison(r)
        torch.cuda.synchronize()
        for r, s in zip(rounds, streams):
            with torch.cuda.stream(s):
                r.run(stream=s)
        torch.cuda.synchronize()
        for r, ref in zip(rounds, refs):
            _same(_snapshot(r), ref)
    # two host threads, each with its own stream
    for r in rounds:
        _poison(r)
    torch.cuda.synchronize()
    errors = []

    def work(r, s):
        try:
            with torch.cuda.stream(s):
                for _ in range(3):
                    r.run(stream=s)
            s.synchronize()
        except Exception as e:  # reported by the main thread
            errors.append(e)

    threads = [threading.Thread(target=work, args=(r, s)) for r, s in zip(rounds, streams)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    torch.cuda.synchronize()
    for r, ref in zip(rounds, refs):
        _same(_snapshot(r), ref)
