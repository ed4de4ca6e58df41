"""The seeded generator: shapes, exact planted counts, reproducibility."""
import numpy as np
import pytest
import torch

from paper_2602_11456_amd import synth


@pytest.mark.parametrize("model,T,N,norm_elems", [
    ("qwen3-4b", 398, 4_022_468_096, 196_096),
    ("qwen3-8b", 399, 8_190_735_360, 308_224),
    ("qwen3-14b", 443, 14_768_307_200, 424_960),
])
def test_tensor_tables(model, T, N, norm_elems):
    table = synth.qwen3_tensor_table(model)
    assert len(table) == T
    assert sum(synth.numel(s) for _, s in table) == N
    assert sum(synth.numel(s) for n, s in table if synth.is_norm(n)) == norm_elems
    names = [n for n, _ in table]
    assert names[0] == "model.embed_tokens.weight"
    assert len(set(names)) == T
    # q, k, v adjacent: their bases equal those of a fused qkv block
    i = names.index("model.layers.0.self_attn.q_proj.weight")
    assert names[i + 1].endswith("k_proj.weight") and names[i + 2].endswith("v_proj.weight")


def test_every_tensor_fits_int32_locally_but_not_globally():
    for model in ("qwen3-4b", "qwen3-8b", "qwen3-14b"):
        table = synth.qwen3_tensor_table(model)
        assert max(synth.numel(s) for _, s in table) - 1 <= 2**31 - 1
        assert sum(synth.numel(s) for _, s in table) - 1 > 2**31 - 1


def test_planted_count_rounding():
    assert synth.planted_count(2048 * 2048, 0.01) == 41_943
    assert synth.planted_count(8_190_735_360, 0.01) == 81_907_354
    assert synth.planted_count(8_190_735_360, 0.001) == 8_190_735
    assert synth.planted_count(100, 0.005) == 1       # 0.5 rounds up
    assert synth.planted_count(0, 0.5) == 0


def test_clustered_plan_numbers():
    hot_rows, H, K, K_hot, K_cold = synth.clustered_plan("qwen3-8b", 0.01)
    assert hot_rows == 99_985
    assert H == 409_538_560
    assert K == 81_907_354
    assert K_hot == 65_525_883
    assert K_cold == 16_381_471


@pytest.mark.parametrize("n,density", [(1, 1.0), (1000, 0.01), (4096, 0.5), (70_001, 0.013)])
def test_pair_planted_exactly(n, density):
    prev, new, pos = synth.make_pair(n, density, seed=5)
    p = prev.view(torch.int16).numpy()
    q = new.view(torch.int16).numpy()
    diff = np.flatnonzero(p != q)
    np.testing.assert_array_equal(diff, pos.numpy())
    assert diff.size == synth.planted_count(n, density)


def test_norm_vector_planting_differs_in_bits():
    prev, new, pos = synth.make_pair(5120, 0.2, seed=1, norm=True)
    assert torch.all(prev == 1.0)
    p = prev.view(torch.int16)
    q = new.view(torch.int16)
    assert int((p != q).sum()) == synth.planted_count(5120, 0.2)


def test_reproducible_and_seed_sensitive():
    a = synth.make_pair(3000, 0.02, seed=42)
    b = synth.make_pair(3000, 0.02, seed=42)
    c = synth.make_pair(3000, 0.02, seed=43)
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x,
                           y.view(torch.int16) if y.dtype == torch.bfloat16 else y)
    assert not torch.equal(a[0].view(torch.int16), c[0].view(torch.int16))


def test_weight_set_subset_matches_full_seeds():
    ws = synth.make_weight_set("qwen3-4b", 0.01, seed=7, tensors=[1, 6, 397])
    assert ws.names == ["model.layers.0.input_layernorm.weight",
                        "model.layers.0.self_attn.q_norm.weight",
                        "model.norm.weight"]
    for p, q, k in zip(ws.prev, ws.new, ws.planted):
        assert int((p.view(torch.int16) != q.view(torch.int16)).sum()) == k
    again = synth.make_weight_set("qwen3-4b", 0.01, seed=7, tensors=[397])
    assert torch.equal(again.new[0].view(torch.int16), ws.new[2].view(torch.int16))


def test_prev_scale():
    prev, _, _ = synth.make_pair(200_000, 0.0, seed=3)
    s = prev.float().std().item()
    assert 0.019 < s < 0.021


@pytest.mark.parametrize("model", ["qwen3-tiny", "qwen3-4b", "qwen3-8b", "qwen3-14b"])
def test_fused_layout_tiles_every_target(model):
    table = synth.qwen3_tensor_table(model)
    targets, sources = synth.qwen3_fused_layout(model)
    assert len(sources) == len(table)
    c = synth.QWEN3[model]
    # per layer 11 tensors become 8 targets
    assert len(targets) == len(table) - 3 * c["layers"]
    blocks = {}
    for (name, shape), (f, off) in zip(table, sources):
        blocks.setdefault(f, []).append((off, synth.numel(shape)))
    for f, (tname, n) in enumerate(targets):
        parts = sorted(blocks[f])
        pos = 0
        for off, size in parts:
            assert off == pos, (tname, parts)
            pos += size
        assert pos == n, tname
    qkv = [n for name, n in targets if name.endswith("qkv_proj.weight")]
    q = c["q_heads"] * c["head_dim"]
    kv = c["kv_heads"] * c["head_dim"]
    assert qkv and all(n == (q + 2 * kv) * c["hidden"] for n in qkv)
