"""The streaming-read probe reads every byte of its buffer exactly once: the
XOR of its sink words equals the XOR of every 32-bit word of the buffer, for
sizes read only by its per-wave streams, only by its tail loop, and by both."""
import numpy as np
import pytest
import torch

from paper_2504_06419_amd import spire
from tests.gpu_helpers import banner

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.mark.parametrize("words", [0, 4, 4 * 1000003, 1 << 24, 4 * (2048 * 1024 + 777)])
def test_probe_reads_every_word_once(words):
    banner(f"hbm read probe: {words} words")
    gen = torch.Generator(device="cpu").manual_seed(words + 7)
    host = torch.randint(-2**31, 2**31 - 1, (words,), generator=gen, dtype=torch.int64).to(torch.int32)
    buf = host.to(DEV)
    sink = torch.full((spire.HBM_PROBE_SINK_WORDS,), -1, dtype=torch.int32, device=DEV)
    spire.hbm_read_probe(buf, sink)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    want = np.bitwise_xor.reduce(host.numpy().view(np.uint32)) if words else np.uint32(0)
    print(f"  xor of sink {got:#010x}, xor of buffer {want:#010x}", flush=True)
    assert got == want
