"""Concurrent callers: several streams fed from one host thread, and several
host threads each with its own stream, all with many host blocks (so every
call also uses the per-device helper stream and its events, shared by all
calls on the device).  Every result equals the same call made alone, bit for
bit."""
import threading

import pytest
import torch

from paper_2512_23068_amd import binding
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu
KW = dict(seg_len=64, chunk_segs=2)


def _problems():
    out = []
    for i, (L, D, K) in enumerate(((1500, 256, 1), (1300, 192, 2), (1700, 128, 1))):
        inp = gu.custom("mamba130m", batch=1, seqlen=L, d_inner=D, n_dirs=K)
        x, dx = gu.inputs_to_dev(inp)
        prm = gu.params_to_dev(inp)
        assert binding.plan(1, L, D, 16, K, **KW)["n_chunks"] > 1
        out.append((x, dx, prm))
    return out


def _refs(probs):
    refs = [binding.scan_jvp(x, dx, prm, **KW) for x, dx, prm in probs]
    torch.cuda.synchronize()
    return refs


def test_several_streams_one_thread():
    probs = _problems()
    refs = _refs(probs)
    streams = [torch.cuda.Stream() for _ in probs]
    outs = [(torch.empty_like(r[0]), torch.empty_like(r[1])) for r in refs]
    for rep in range(3):
        for o in outs:
            o[0].fill_(1.0)
            o[1].fill_(1.0)
        torch.cuda.synchronize()
        for (x, dx, prm), st, o in zip(probs, streams, outs):   # enqueued back to back, run concurrently
            binding.scan_jvp(x, dx, prm, out=o, stream=st, **KW)
        torch.cuda.synchronize()
        for o, r in zip(outs, refs):
            assert torch.equal(o[0], r[0]) and torch.equal(o[1], r[1]), rep


def test_several_host_threads():
    probs = _problems()
    refs = _refs(probs)
    errors = []

    def work(i):
        try:
            x, dx, prm = probs[i]
            st = torch.cuda.Stream()
            o = (torch.empty_like(refs[i][0]), torch.empty_like(refs[i][1]))
            for rep in range(4):
                binding.scan_jvp(x, dx, prm, out=o, stream=st, **KW)
                st.synchronize()
                if not (torch.equal(o[0], refs[i][0]) and torch.equal(o[1], refs[i][1])):
                    errors.append((i, rep))
        except Exception as e:   # reported by the main thread
            errors.append((i, repr(e)))

    threads = [threading.Thread(target=work, args=(i,)) for i in range(len(probs))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads)
    assert not errors, errors
