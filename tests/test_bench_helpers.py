"""Host-side helpers of bench.py (CPU)."""
import numpy as np

import bench
from oracle_pins import llama_config


def test_llama3_frequencies_match_hugging_face():
    """The Llama-3 rotation frequencies the benchmark feeds both the GPU and
    the oracle agree with Hugging Face's Llama rotary module (both are fp32;
    they may differ in the last bit of the blend)."""
    from transformers.models.llama.modeling_llama import LlamaRotaryEmbedding
    hf = LlamaRotaryEmbedding(llama_config(32, 8, 128)).inv_freq.numpy()
    mine = bench.llama3_rope_inv_freq()
    assert mine.dtype == np.float32 and mine.shape == (64,)
    assert np.abs(hf / mine - 1.0).max() < 1e-6
    plain = bench.LLAMA_ROPE_THETA ** (-np.arange(0, 128, 2) / 128.0)
    assert (mine[:8] == plain[:8].astype(np.float32)).all()   # kept
    assert np.allclose(mine[-4:], plain[-4:] / 32.0, rtol=1e-6)  # slowed
