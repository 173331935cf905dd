"""The ceiling probes on the device: rates that are positive and below the
part's published peaks (dense bf16 MFMA 2.5 PFLOP/s at the 2.4 GHz peak
clock, HBM3E 8 TB/s), and argument checks that need a real buffer."""
import numpy as np
import pytest

from paper_2608_14575_amd import hwr

pytestmark = pytest.mark.gpu


def test_mfma_ceiling_is_below_the_published_peak():
    hwr.load()
    for w in (1, 2):
        t, mhz = hwr.hwr_probe_mfma_bf16(0, w, 1024, 3)
        print(f"[probe] mfma bf16, {w} wave(s) per SIMD: {t:.0f} TFLOP/s at {mhz:.0f} MHz", flush=True)
        assert 500.0 < t <= 2500.0
        # within the part's clock range; and at most what the clock allows
        # (1024 SIMDs, 32768 flops per 32-cycle product)
        assert 500.0 < mhz <= 2500.0
        assert t <= 1024 * 1024 * mhz * 1e6 / 1e12 * 1.02


def test_hbm_ceilings_are_below_the_published_peak():
    import torch
    hwr.load()
    nbytes = 1 << 30
    buf = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda:0")
    # 1 GiB is four times the last-level cache: at most a quarter of it can
    # be served from there
    for w in (2, 8):
        g = hwr.hwr_probe_hbm_read(0, buf.data_ptr(), nbytes, w, 3)
        print(f"[probe] hbm read 1 GiB, {w} waves per SIMD: {g:.0f} GB/s", flush=True)
        assert 1000.0 < g < 8000.0 * 1.35
    # a length that is not a whole number of 16-byte pieces, a misaligned start
    for probe in (hwr.hwr_probe_hbm_read, hwr.hwr_probe_hbm_write):
        with pytest.raises(hwr.HwrError):
            probe(0, buf.data_ptr(), 1000, 2, 3)
        with pytest.raises(hwr.HwrError):
            probe(0, buf.data_ptr() + 4, 1 << 20, 2, 3)
    # the read probe only reads; rejected calls write nothing
    assert bool((buf == 1).all())
    for w in (1, 4):
        g = hwr.hwr_probe_hbm_write(0, buf.data_ptr(), nbytes, w, 3)
        print(f"[probe] hbm write 1 GiB, {w} waves per SIMD: {g:.0f} GB/s", flush=True)
        assert 1000.0 < g < 8000.0 * 1.35
    # the write probe stays inside its buffer: a guard after it is untouched
    torch.cuda.synchronize()
    big = torch.zeros(nbytes // 4 + 1024, dtype=torch.int32, device="cuda:0")
    hwr.hwr_probe_hbm_write(0, big.data_ptr(), nbytes, 2, 1)
    assert bool((big[nbytes // 4:] == 0).all())
    assert bool((big[:nbytes // 4] != 0).any())


def test_launch_floor_plain_and_graph():
    hwr.load()
    for graph in (False, True):
        p50, p99 = hwr.hwr_probe_launch_floor(0, graph, 500)
        print(f"[probe] launch floor ({'graph' if graph else 'plain'} launch): p50 {p50:.1f} us, p99 {p99:.1f} us",
              flush=True)
        assert 0.5 < p50 <= p99 < 10_000.0


def _bf16_bits(f32: np.ndarray) -> np.ndarray:
    """bf16 bits of fp32 values, nearest with ties to even (finite inputs)."""
    u = f32.view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def test_feature_log_gives_the_features_of_the_exact_log():
    """The device's feature logarithm against numpy's fp64 log on 4M
    arguments over every feature's range (input lengths and queue counts
    plus one, up to 2^31; parameter counts in billions; latencies in
    seconds): relative error below 2^-48, and every feature value (ln times
    its scale, rounded to fp32, then to bf16) the same."""
    rng = np.random.default_rng(7)
    n = 1 << 20
    cases = {
        "input length": (1.0 + rng.integers(0, 40000, n).astype(np.float64), 0.125),
        "1 + queue": (1.0 + rng.integers(0, 1 << 31, n).astype(np.float64), 0.5),
        "params (B)": (np.exp(rng.uniform(-1, 11, n)).astype(np.float32).astype(np.float64), 0.25),
        "seconds": (np.exp(rng.uniform(-12, 8, n)).astype(np.float32).astype(np.float64), 0.25),
    }
    for name, (x, scale) in cases.items():
        y = hwr.hwr_probe_feature_log(0, x)
        ref = np.log(x)
        rel = np.abs(y - ref) / np.maximum(np.abs(ref), 1e-300)
        rel[ref == 0] = np.abs(y[ref == 0])
        f_dev = (y * scale).astype(np.float32)
        f_ref = (ref * scale).astype(np.float32)
        n32 = int((f_dev != f_ref).sum())
        n16 = int((_bf16_bits(f_dev) != _bf16_bits(f_ref)).sum())
        print(f"[probe] feature log, {name}: max rel {rel.max():.2e}, fp32 differ {n32}, bf16 differ {n16}",
              flush=True)
        assert rel.max() < 2.0 ** -48, name
        assert n16 == 0, name
