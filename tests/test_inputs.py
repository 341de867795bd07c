"""The seeded input generators are deterministic and have the stated shape
and outlier structure (no method arithmetic is involved)."""
import torch

from paper_2607_01831_amd import inputs


def test_deterministic_and_shaped():
    w = inputs.WORKLOADS["tiny-gqa2-4k"]
    a = inputs.kv(w, "k", T=300)
    b = inputs.kv(w, "k", T=300)
    assert a.dtype == torch.bfloat16 and a.shape == (300, w.Hkv, 128)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    v = inputs.kv(w, "v", T=300)
    assert not torch.equal(a, v)


def test_outlier_columns():
    w = inputs.WORKLOADS["tiny-gqa2-4k"]
    m = inputs.outlier_columns(w, 0)
    assert m.shape == (4, 128) and (m.sum(dim=1) == 4).all()
    w2 = inputs.WORKLOADS["llama3-8b-32k"]
    m2 = inputs.outlier_columns(w2, 3)
    assert int(m2.sum()) == round(0.01 * 8 * 128) == 10
    k = inputs.kv(w, "k", T=4096).float()
    big = k.abs().amax(dim=0)[m].min()
    small = k.abs().amax(dim=0)[~m].max()
    assert big > 2 * small  # the x10 columns stand out over 4096 tokens


def test_paged_block_table_is_a_permutation():
    w = inputs.WORKLOADS["paged-b16-16k-64k"]
    lens = inputs.seq_lengths(w)
    assert lens.shape == (16,) and int(lens.min()) >= 16384 and int(lens.max()) <= 65536
    table, n_blocks = inputs.paged_block_table(lens, 16, inputs.seed_of(w.wid, inputs.T_BLOCKS))
    used = torch.cat([table[b, : -(-int(t) // 16)] for b, t in enumerate(lens)])
    assert used.numel() == n_blocks
    assert torch.equal(used.sort().values, torch.arange(n_blocks, dtype=torch.int32))
