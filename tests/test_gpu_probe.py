"""The ceiling probes on the device: rates that are positive and below the
part's published peaks (dense bf16 MFMA 2.5 PFLOP/s at the 2.4 GHz peak
clock, HBM3E 8 TB/s), and argument checks that need a real buffer."""
import pytest

from paper_2608_14575_amd import hwr

pytestmark = pytest.mark.gpu


def test_mfma_ceiling_is_below_the_published_peak():
    hwr.load()
    for w in (1, 2):
        t = hwr.hwr_probe_mfma_bf16(0, w, 1024, 3)
        print(f"[probe] mfma bf16, {w} wave(s) per SIMD: {t:.0f} TFLOP/s", flush=True)
        assert 500.0 < t <= 2500.0


def test_hbm_read_ceiling_is_below_the_published_peak():
    import torch
    hwr.load()
    nbytes = 1 << 30
    buf = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda:0")
    for w in (2, 8):
        g = hwr.hwr_probe_hbm_read(0, buf.data_ptr(), nbytes, w, 3)
        print(f"[probe] hbm read 1 GiB, {w} waves per SIMD: {g:.0f} GB/s", flush=True)
        # 1 GiB is four times the last-level cache: at most a quarter of it
        # can be served from there
        assert 1000.0 < g < 8000.0 * 1.35
    # a length that is not a whole number of 16-byte pieces, a misaligned start
    with pytest.raises(hwr.HwrError):
        hwr.hwr_probe_hbm_read(0, buf.data_ptr(), 1000, 2, 3)
    with pytest.raises(hwr.HwrError):
        hwr.hwr_probe_hbm_read(0, buf.data_ptr() + 4, 1 << 20, 2, 3)
    # the probe only reads
    assert bool((buf == 1).all())
