"""The seeded input generator: determinism and the structure the kernels rely on."""
import numpy as np
import torch

import cw_workloads as cw


def test_deterministic_and_thread_independent():
    a = cw.materialize(cw.custom_spec([40, 9], [7, 30], num_kv_heads=2, gqa_group=2, head_dim=16,
                                      page_size=8, seed=5), threads=1)
    b = cw.materialize(cw.custom_spec([40, 9], [7, 30], num_kv_heads=2, gqa_group=2, head_dim=16,
                                      page_size=8, seed=5), threads=4)
    for x, y in ((a.q, b.q), (a.k_pool, b.k_pool), (a.v_new, b.v_new), (a.block_table, b.block_table)):
        assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x,
                           y.view(torch.int16) if y.dtype == torch.bfloat16 else y)


def test_named_specs():
    t = cw.spec_for("turn")
    assert t.flops() == 4 * 128 * 32 * (1024 * 16384 + 1024 * 1025 // 2)
    assert round(t.flops() / 1e9, 2) == 283.48
    lg = cw.spec_for("long")
    assert lg.attention_pairs() == 1107300352
    b = cw.spec_for("batch16")
    assert b.num_seqs == 16 and b.prefix_lens.min() >= 8192 and b.prefix_lens.max() <= 65536
    assert b.suffix_lens.min() >= 200 and b.suffix_lens.max() <= 4000
    m = cw.spec_for("mixed")
    assert (m.suffix_lens == 1).sum() == 48
    ext = m.suffix_lens > 1
    assert m.suffix_lens[ext].min() >= 256 and m.suffix_lens[ext].max() <= 2048
    assert m.prefix_lens[ext].min() >= 8192 and m.prefix_lens[~ext].min() >= 2048
    assert m.kv_dtype == "fp8"
    c = cw.spec_for("chunked")
    dec = c.suffix_lens == 1
    assert dec.sum() == 32 and (~dec).sum() == 32
    assert c.suffix_lens[~dec].min() >= 128 and c.suffix_lens[~dec].max() <= 512
    assert c.prefix_lens[~dec].min() >= 8192 and c.prefix_lens.max() <= 32768
    assert c.prefix_lens[dec].min() >= 2048 and c.kv_dtype == "bf16"


def test_block_table_and_sentinels():
    spec = cw.custom_spec([24, 24, 37], [5, 9, 3], num_kv_heads=1, gqa_group=1, head_dim=8,
                          page_size=8, seed=2, shared_prefix_tokens=16)
    w = cw.materialize(spec, threads=1)
    bt = w.block_table.numpy()
    need = spec.pages_needed()
    assert np.all(bt[:, :2] == bt[0, :2])  # shared prefix pages are the same physical pages
    used = []
    for b in range(3):
        assert np.all(bt[b, need[b]:] == cw.BT_UNUSED)
        used += bt[b, 2 if b else 0:need[b]].tolist()
    assert len(set(used)) == len(used)  # private pages are not shared
    assert max(used) < spec.num_pages
    bits = w.k_pool.view(torch.int16).numpy().view(np.uint16)
    for b in range(3):
        lp = int(spec.prefix_lens[b])
        for j in range(need[b] * 8):
            pg, sl = bt[b, j // 8], j % 8
            is_nan = np.all(bits[pg, :, sl] == cw.BF16_NAN_BITS)
            assert is_nan == (j >= lp)  # prefix slots hold data, every other slot NaN
    unused = sorted(set(range(spec.num_pages)) - set(used))
    assert np.all(bits[unused] == cw.BF16_NAN_BITS)
