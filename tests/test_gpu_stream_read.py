"""The streaming-read calibration kernel (santa_stream_read): every byte of the
buffer is read exactly once, checked by the XOR fold of the sink against numpy's
XOR over the same words, on sizes that split unevenly over the workgroups."""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2605_01910_amd import santa as S

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n_words", [4, 4 * 2047, 4 * 2049 + 4 * 37, (64 << 20) // 4 + 4 * 999, (600 << 20) // 4 + 4 * 3])
def test_stream_read_folds_every_word(n_words):
    rng = np.random.default_rng(n_words)
    host = rng.integers(0, 2**32, size=n_words, dtype=np.uint32)
    buf = torch.from_numpy(host.view(np.int32)).cuda()
    sink = torch.zeros(S.STREAM_READ_GROUPS, dtype=torch.int32, device="cuda")
    S.santa_stream_read(buf, sink)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(host)


def test_stream_read_timed_with_call_events():
    buf = torch.ones((8 << 20) // 4, dtype=torch.float32, device="cuda")
    sink = torch.empty(S.STREAM_READ_GROUPS, dtype=torch.int32, device="cuda")
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(); b.record()
    torch.cuda.synchronize()
    S.santa_time_next_call(a, b)
    S.santa_stream_read(buf, sink)
    torch.cuda.synchronize()
    us = a.elapsed_time(b) * 1e3
    assert 0.0 < us < 10000.0
