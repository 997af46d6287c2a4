"""GPU check of the streaming-read probes (measurement support, not a step
of the method): every thread of the probe folds the 16-byte words it reads
into an XOR and writes it to its sink slot, so a host walk of the same
grid-stride assignment reproduces the sink exactly -- which shows the probe
reads every byte of its range once and nothing beyond it.  The series form
writes the last piece's result last."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

wf = pytest.importorskip("paper_2606_07710_amd")
DEV = "cuda"
THREADS = 256


def _expected(words, wgs, depth):
    """Sink of one probe over `words` ([n16, 4] uint32): word j belongs to
    the thread whose piece of its round holds it."""
    n16 = words.shape[0]
    piece = THREADS * depth
    off = np.arange(n16) % (wgs * piece)
    owner = (off // piece) * THREADS + (off % piece) % THREADS
    out = np.zeros((wgs * THREADS, 4), np.uint32)
    np.bitwise_xor.at(out, owner, words)
    return out


def _data(n16, seed):
    g = np.random.default_rng(seed)
    return g.integers(0, 2**32, size=(n16, 4), dtype=np.uint32)


@pytest.mark.parametrize("n16,wgs", [(1, 1), (4096, 2), (37 * 1000 + 13, 5), (1 << 16, 16)])
def test_read_probe_sink(n16, wgs):
    words = _data(n16, n16)
    src = torch.from_numpy(words.view(np.uint8).reshape(-1).copy()).to(DEV)
    sink = torch.zeros(wgs * 4096, dtype=torch.uint8, device=DEV)
    wf.wf_read_probe(src, sink, wgs)
    torch.cuda.synchronize()
    got = sink.cpu().numpy().view(np.uint32).reshape(-1, 4)[: wgs * THREADS]
    np.testing.assert_array_equal(got, _expected(words, wgs, 8))


@pytest.mark.parametrize("depth", [4, 8])
@pytest.mark.parametrize("n16,n_bufs,reps,wgs", [(5000, 3, 2, 3), (1 << 14, 1, 1, 8)])
def test_read_probe_series_sink(depth, n16, n_bufs, reps, wgs):
    words = _data(n16 * n_bufs, 7 + depth)
    buf = torch.from_numpy(words.view(np.uint8).reshape(-1).copy()).to(DEV)
    sink = torch.zeros(wgs * 4096, dtype=torch.uint8, device=DEV)
    wf.wf_read_probe_series(buf, n16 * 16, n_bufs, reps, sink, wgs, depth)
    torch.cuda.synchronize()
    got = sink.cpu().numpy().view(np.uint32).reshape(-1, 4)[: wgs * THREADS]
    np.testing.assert_array_equal(got, _expected(words[(n_bufs - 1) * n16:], wgs, depth))
