"""The engine's peak microbenchmarks (HBM read bandwidth, 32x32x16 bf16 MFMA
throughput), called through the C ABI: plausible values for an MI355X
(published peaks 8 TB/s and 2.5 PFLOP/s dense bf16), and the argument checks."""
import pytest

from moa_inputs import CONFIGS
from moa_inputs.configs import EngineConsts
from paper_2606_03014_amd import Engine
from paper_2606_03014_amd import moa as M

pytestmark = pytest.mark.gpu


def test_measured_peaks_are_plausible():
    c = CONFIGS["tiny-moa-fp32"]
    # 16,384 blocks of 64 KiB: a 1 GiB KV pool to read; 64 rows x 4096 logits of scratch
    consts = EngineConsts(num_kv_blocks=16384, max_num_seqs=64, max_prefill_tokens=64, max_model_len=256)
    eng = Engine(c.model, "f32", consts, 1)
    try:
        read_bps, mfma_fps = eng.measure_peaks()
    finally:
        eng.close()
    print(f"HBM read {read_bps / 1e12:.2f} TB/s, bf16 MFMA {mfma_fps / 1e15:.2f} PFLOP/s", flush=True)
    assert 2e12 < read_bps < 8.5e12
    assert 0.8e15 < mfma_fps < 2.6e15


def test_measure_peaks_rejects_a_small_pool():
    c = CONFIGS["tiny-moa-fp32"]
    consts = EngineConsts(num_kv_blocks=128, max_num_seqs=64, max_prefill_tokens=64, max_model_len=256)
    eng = Engine(c.model, "f32", consts, 1)
    try:
        with pytest.raises(M.MoaError):
            eng.measure_peaks()
    finally:
        eng.close()
