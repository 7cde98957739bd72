"""The matrix-core reference loop behind libra_mfma_loop: it runs on the GPU,
records a plausible shader clock, and its throughput lies below the published
dense bf16 peak (and well above a tenth of it)."""
import pytest

import paper_2607_23250_amd as pl

PUBLISHED_BF16_TFLOPS = 2516.6


def test_rejects_bad_arguments_without_a_gpu():
    with pytest.raises(pl.LibraError) as e:
        pl.libra_mfma_loop_size(3)
    assert e.value.code == pl.LIBRA_EINVAL


@pytest.mark.gpu
@pytest.mark.parametrize("wps", [1, 2])
def test_loop_throughput_and_clock(wps):
    import torch
    dev = torch.device("cuda:0")
    words, prods = pl.libra_mfma_loop_size(wps)
    assert words == 3 * prods // (16 * wps) and prods % (16 * wps) == 0
    rec = torch.zeros(words, dtype=torch.int64, device=dev)
    with pytest.raises(pl.LibraError):
        pl.libra_mfma_loop(wps, 10, rec[: words - 1])
    iters = 20000
    pl.libra_mfma_loop(wps, 100, rec)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s = torch.cuda.current_stream(dev)
    e0.record(s)
    pl.libra_mfma_loop(wps, iters, rec)
    e1.record(s)
    e1.synchronize()
    ms = e0.elapsed_time(e1)
    r = rec.view(-1, 3).cpu().numpy()
    assert (r[:, 0] > 0).all() and (r[:, 1] > 0).all()
    ghz = r[:, 0].sum() / r[:, 1].sum() * 0.1
    tf = 32768.0 * iters * prods / (ms * 1e-3) / 1e12
    print(f"waves/SIMD {wps}: {tf:.1f} TFLOP/s at {ghz:.3f} GHz")
    assert 0.5 < ghz < 2.6
    assert 0.1 * PUBLISHED_BF16_TFLOPS < tf < 1.02 * PUBLISHED_BF16_TFLOPS
