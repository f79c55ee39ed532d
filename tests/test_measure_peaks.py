"""The measurement helpers that benchmarks report beside the vendor peaks: the read kernel
folds every 32-bit word of its buffer into its checksum words (so none of its loads is
dropped or duplicated, whatever the size and tail), and the matrix-core loop leaves its
exact value in every lane.  They compute nothing of the method; this checks that what
they time is the work they claim."""
import numpy as np
import pytest
import torch

from paper_2607_07409_amd import binding as b

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("nbytes", [16, 4096 + 48, (1 << 20) + 16, (33 << 20) + 208, 64 << 20])
def test_read_checksum_is_the_xor_of_the_buffer(nbytes):
    print(f"measure_read nbytes={nbytes}", flush=True)
    g = np.random.default_rng(nbytes)
    host = g.integers(0, 1 << 32, size=nbytes // 4, dtype=np.uint64).astype(np.uint32)
    # guard words on both sides: they must not enter the checksum
    pad = np.full(64, 0xDEADBEEF, dtype=np.uint32)
    dev = torch.from_numpy(np.concatenate([pad, host, pad]).view(np.int32)).to("cuda")
    view = dev[64:64 + host.size]
    words = b.measure_read(view)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(words.cpu().numpy().view(np.uint32))
    assert int(got) == int(np.bitwise_xor.reduce(host))
    assert words.numel() == b.MEASURE_READ_WORDS
    # each workgroup folds a fixed stride of the buffer: repeat calls give the same words
    again = b.measure_read(view).cpu()
    assert torch.equal(again, words.cpu())


@pytest.mark.parametrize("groups,iters,x", [(1, 1, 1.0), (7, 33, 0.5), (300, 1000, 1.0 / 64),
                                            (2048, 64, 2.0 ** -20)])
def test_mfma_loop_value_is_exact(groups, iters, x):
    print(f"measure_mfma groups={groups} iters={iters} x={x}", flush=True)
    out = b.measure_mfma(groups, iters, x, device="cuda")
    torch.cuda.synchronize()
    assert out.numel() == groups * 256
    expect = iters * 1024.0 * x * x
    assert torch.all(out == expect), (out.min().item(), out.max().item(), expect)
