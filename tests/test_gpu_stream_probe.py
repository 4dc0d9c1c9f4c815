"""The reference streams of zf_measure.h (measurement only): the copy
leaves dst equal to src, the read-modify-write pass leaves every 32-bit word
xor key, and the read pass writes nothing unless its folded data equal the
key -- on sizes with a ragged last block (not a multiple of the 4 KiB block
chunk) and buffers padded with sentinels that must stay intact."""
import pytest
import torch

pytestmark = pytest.mark.gpu

zf = pytest.importorskip("paper_2505_12242_amd")

SIZES = [16, 4096, 4096 + 16, 8192 + 16, 3 * 2**20 + 48, 64 * 2**20]
PAD = 4096


@pytest.mark.parametrize("nbytes", SIZES)
def test_probe_streams(nbytes):
    g = torch.Generator(device="cuda").manual_seed(nbytes)
    src_buf = torch.randint(0, 256, (nbytes + 2 * PAD,), dtype=torch.uint8, device="cuda",
                            generator=g)
    dst_buf = torch.randint(0, 256, (nbytes + 2 * PAD,), dtype=torch.uint8, device="cuda",
                            generator=g)
    src, dst = src_buf[PAD:PAD + nbytes], dst_buf[PAD:PAD + nbytes]
    src0, dst0 = src_buf.clone(), dst_buf.clone()
    zf.stream_probe(zf.PROBE_COPY, src, dst, nbytes)
    torch.cuda.synchronize()
    assert torch.equal(dst, src)
    assert torch.equal(src_buf, src0)
    assert torch.equal(dst_buf[:PAD], dst0[:PAD]) and torch.equal(dst_buf[PAD + nbytes:],
                                                                  dst0[PAD + nbytes:])
    key = 0x9E3779B9
    before = dst_buf.clone()
    zf.stream_probe(zf.PROBE_RMW, None, dst, nbytes, key=key)
    torch.cuda.synchronize()
    want = (before[PAD:PAD + nbytes].view(torch.int32) ^ torch.tensor(key, dtype=torch.int64)
            .to(torch.int32).cuda()).view(torch.uint8)
    assert torch.equal(dst, want)
    assert torch.equal(dst_buf[:PAD], before[:PAD])
    assert torch.equal(dst_buf[PAD + nbytes:], before[PAD + nbytes:])
    sink = torch.full((4,), 7, dtype=torch.int32, device="cuda")
    zf.stream_probe(zf.PROBE_READ, src, sink, nbytes, key=0x12345678)
    torch.cuda.synchronize()
    # the folded value of random data is (overwhelmingly likely) not the key
    assert torch.equal(sink, torch.full((4,), 7, dtype=torch.int32, device="cuda"))
