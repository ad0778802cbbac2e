"""bd_decode_static (the decode that allocates nothing, its state in the
library's static scratch) against bd_decode through the C ABI: identical
tokens, commit steps and forwards on two calls in a row, the second with a
smaller input (fewer sequences, a shorter prompt and generation), so the
second call runs on scratch the first one left behind; and the size check
that refuses a decode whose state does not fit."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from bd_synth import Workload, make_weights, make_prompts   # noqa: E402


def _model(w):
    from paper_2609_33887_amd import bd
    return bd.Model(w, make_weights(w))


W_BF16 = Workload("static_gqa", 110, n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, head_dim=128,
                  ffn_dim=512, vocab=1024, dtype="bf16", batch=4, prompt_len=64, block_size=16,
                  n_inflight=2, gen_len=64)
W_MOE = Workload("static_moe", 111, n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, head_dim=128,
                 ffn_dim=0, vocab=1024, dtype="bf16", batch=3, prompt_len=32, block_size=16, n_inflight=2,
                 gen_len=48, n_experts=8, top_k=2, expert_ffn=128, n_shared=1)
W_F32 = Workload("static_f32", 112, n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64,
                 ffn_dim=512, vocab=1024, dtype="f32", batch=2, prompt_len=16, block_size=8, n_inflight=2,
                 gen_len=32)


@pytest.mark.parametrize("w", [W_BF16, W_MOE, W_F32], ids=lambda w: w.name)
def test_static_decode_matches_decode_twice(w):
    from paper_2609_33887_amd import bd
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    model = _model(w)
    prompts = make_prompts(w)
    B = w.block_size
    calls = [(prompts, w.gen_len, 0.9), (prompts[:-1, :w.prompt_len - B], w.gen_len - B, 0.8)]
    for pr, G, tau in calls:
        print(f"[static] {w.name} b={pr.shape[0]} P={pr.shape[1]} G={G} tau={tau}", flush=True)
        ref = bd.decode(model, pr, G, tau, w.n_inflight, B)
        got = bd.decode(model, pr, G, tau, w.n_inflight, B, static=True)
        for a, b in zip(ref, got):
            np.testing.assert_array_equal(a, b)
    model.close()


def test_static_decode_refuses_a_state_beyond_the_scratch():
    from paper_2609_33887_amd import bd
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w = W_BF16
    model = _model(w)
    prompts = make_prompts(w, 64)     # 64 sequences x 128 positions x 2 layers of K/V pairs and more
    big = np.tile(prompts, (1, 16))   # prompts of 1024 tokens
    with pytest.raises(bd.BDError) as e:
        bd.decode(model, big, w.gen_len, 0.9, w.n_inflight, w.block_size, static=True)
    assert e.value.status == bd.BD_EUNSUPPORTED and "scratch" in str(e.value)
    # the refusal leaves the scratch usable
    ref = bd.decode(model, prompts[:2], w.gen_len, 0.9, w.n_inflight, w.block_size)
    got = bd.decode(model, prompts[:2], w.gen_len, 0.9, w.n_inflight, w.block_size, static=True)
    for a, b in zip(ref, got):
        np.testing.assert_array_equal(a, b)
    model.close()
