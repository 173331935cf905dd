"""The binding checks every buffer of a route call (kind, contiguity,
memory space, size) before the library sees a pointer: a short, strided or
misplaced buffer raises HwrError(HWR_ERR_INVALID_ARG) instead of reaching the
kernels.  No device and no library call needed."""
import numpy as np
import pytest

from paper_2608_14575_amd import hwr

SHAPE = dict(n=5, D=64, M=3, N=4, K=1, dtype="bf16", n_heads=2, device=0)


def _host(n=5, D=64, M=3, N=4):
    return dict(emb=np.zeros((n, D), np.uint16), input_len=np.ones(n, np.int32),
                expected_out_len=np.ones(n, np.int32), slo_s=np.ones(n, np.float32),
                choice=np.zeros(n, np.int32), feasible=np.zeros(n, np.uint8), utility=np.zeros(n, np.float32),
                cand_ttft=np.zeros((n, N), np.float32), cand_quality=np.zeros((n, M), np.float32))


def _raises(msg, **bufs):
    with pytest.raises(hwr.HwrError) as e:
        hwr.check_batch(**SHAPE, **bufs)
    assert e.value.status == hwr.HWR_ERR_INVALID_ARG
    assert msg in str(e.value)


def test_valid_host_batch_passes():
    hwr.check_batch(**SHAPE, mem=hwr.HWR_MEM_HOST, **_host())


def test_host_batch_errors():
    b = _host()
    _raises("emb: 256 elements, needs 320", mem=hwr.HWR_MEM_HOST, **{**b, "emb": b["emb"][:4]})
    _raises("input_len: dtype int64", mem=hwr.HWR_MEM_HOST, **{**b, "input_len": np.ones(5, np.int64)})
    _raises("choice: not contiguous", mem=hwr.HWR_MEM_HOST, **{**b, "choice": np.zeros(10, np.int32)[::2]})
    _raises("cand_ttft: 16 elements, needs 20", mem=hwr.HWR_MEM_HOST, **{**b, "cand_ttft": np.zeros((4, 4), np.float32)})
    _raises("cand_quality: 12 elements, needs 15", mem=hwr.HWR_MEM_HOST,
            **{**b, "cand_quality": np.zeros((4, 3), np.float32)})
    _raises("expected_out_len", mem=hwr.HWR_MEM_HOST, **{**b, "expected_out_len": None})
    _raises("unknown mem", mem=7, **b)


def test_three_heads_may_omit_output_length():
    b = _host()
    b["expected_out_len"] = None
    hwr.check_batch(**{**SHAPE, "n_heads": 3}, mem=hwr.HWR_MEM_HOST, **b)


def test_device_batch_rejects_host_and_meta_buffers():
    torch = pytest.importorskip("torch")
    b = _host()
    _raises("emb: a device batch needs device tensors", mem=hwr.HWR_MEM_DEVICE, **b)
    tb = {k: torch.from_numpy(v.view(np.int16) if v.dtype == np.uint16 else v) for k, v in b.items()}
    _raises("emb: on cpu, expected cuda:0", mem=hwr.HWR_MEM_DEVICE, **tb)
    meta = {k: torch.empty(v.shape, dtype=v.dtype, device="meta") for k, v in tb.items()}
    _raises("emb: on meta, expected cuda:0", mem=hwr.HWR_MEM_DEVICE, **meta)


def test_host_batch_accepts_cpu_tensors_and_checks_them():
    torch = pytest.importorskip("torch")
    b = _host()
    tb = {k: torch.from_numpy(v.view(np.int16) if v.dtype == np.uint16 else v) for k, v in b.items()}
    hwr.check_batch(**SHAPE, mem=hwr.HWR_MEM_HOST, **tb)
    _raises("utility: dtype torch.float64", mem=hwr.HWR_MEM_HOST,
            **{**tb, "utility": torch.zeros(5, dtype=torch.float64)})
    _raises("cand_ttft: not contiguous", mem=hwr.HWR_MEM_HOST,
            **{**tb, "cand_ttft": torch.zeros((4, 5), dtype=torch.float32).t()})


def test_several_weights_need_n_times_k_outputs():
    b = _host()
    with pytest.raises(hwr.HwrError) as e:
        hwr.check_batch(**{**SHAPE, "K": 3}, mem=hwr.HWR_MEM_HOST, **b)
    assert "choice: 5 elements, needs 15" in str(e.value)
