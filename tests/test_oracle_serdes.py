"""Pins for the oracle's serializer / deserializer, CPU only.

Sec. 4.2 and Sec. 5: the serializer writes an object's packed Anchor stream
followed immediately by its shared scalars into one contiguous transmission
buffer and the Residual stream into another; the deserializer scatters the
Anchor buffer into the KV pages (Anchor phase) and later combines the
Residual buffer with those Anchors into the 8-bit codes (Residual phase).

Pinned by: section offsets stated by hand; a whole buffer written out by hand
for a one-token object (the G1 row of the codec goldens); and round trips
against the whole-sequence encode and merge of the oracle (which have pins of
their own), with objects delivered in shuffled order into a paged pool.
"""
import numpy as np
import pytest

import oracle
from tests._util import bf16_bits

HEAD_DIM = 128


def test_sections_stated_by_hand():
    # one kv head, 130 tokens: two K groups (128 + 2 tokens)
    s = oracle.serialized_sections(1, 130)
    assert s["k_anc"] == (0, 130 * 64)
    assert s["v_anc"] == (8320, 8320)
    assert s["k_scale"] == (16640, 2 * 128 * 4)
    assert s["k_zero"] == (17664, 1024)
    assert s["v_scale"] == (18688, 130 * 4)
    assert s["v_zero"] == (19208, 520)
    assert s["anchor_bytes"] == 19728
    assert s["k_res"] == (0, 8320) and s["v_res"] == (8320, 8320)
    assert s["residual_bytes"] == 16640
    # a 32K-token layer of 8 kv heads: the anchor buffer is the 144 bytes per
    # token per kv head the anchor decode reads (64 + 64 nibbles, 8 V metadata,
    # 1024 K-metadata bytes per 128 tokens)
    s = oracle.serialized_sections(8, 32768)
    assert s["anchor_bytes"] == 144 * 32768 * 8
    assert s["residual_bytes"] == 128 * 32768 * 8


def test_one_token_object_written_out_by_hand():
    # K row = V row = [0, 255, 126.5, 2.5, 0 x 124] (all exact in BF16).
    row = np.zeros(HEAD_DIM, np.float32)
    row[:4] = [0.0, 255.0, 126.5, 2.5]
    bits = bf16_bits(row).reshape(1, 1, HEAD_DIM)
    anc, res = oracle.serialize(1, 1, bits, bits)
    assert anc.size == 64 + 64 + 512 + 512 + 4 + 4 and res.size == 128
    # K: each channel's group holds one token -> range 0 -> scale 0, zero = the
    # value, code 0: anchor and residual rows are all zero
    assert not anc[0:64].any() and not res[0:64].any()
    # V: the token's group is [0, 255] -> scale 1, zero 0, codes 0, 255, 126
    # (126.5 rounds half to even), 2: anchors 0, 15, 7, 0 -> bytes 0xF0, 0x07;
    # residuals 0, 15, 14, 2 -> bytes 0xF0, 0x2E (low nibble = even dim)
    want_va = np.zeros(64, np.uint8)
    want_va[:2] = [0xF0, 0x07]
    want_vr = np.zeros(64, np.uint8)
    want_vr[:2] = [0xF0, 0x2E]
    assert np.array_equal(anc[64:128], want_va)
    assert np.array_equal(res[64:128], want_vr)
    # K scales (128 zeros), K zeros (the row itself), V scale 1, V zero 0
    assert np.array_equal(anc[128:640].view(np.float32), np.zeros(HEAD_DIM, np.float32))
    assert np.array_equal(anc[640:1152].view(np.float32), row)
    assert anc[1152:1156].view(np.float32)[0] == 1.0
    assert anc[1156:1160].view(np.float32)[0] == 0.0


def _sequence(T, Hkv, seed):
    rng = np.random.default_rng(seed)
    k = rng.standard_normal((T, Hkv, HEAD_DIM)).astype(np.float32)
    k[:, :, 5] *= 9.0  # an outlier channel
    v = rng.standard_normal((T, Hkv, HEAD_DIM)).astype(np.float32)
    return bf16_bits(k), bf16_bits(v)


def _paged_pool(T, Hkv, bt, max_tokens, seed):
    n_blocks = -(-max_tokens // bt) + 3
    rng = np.random.default_rng(seed)
    table = rng.permutation(n_blocks)[: -(-max_tokens // bt)].astype(np.int32).reshape(1, -1)
    L = oracle.Layout(Hkv=Hkv, bt=bt, max_blocks=table.shape[1], max_tokens=max_tokens)
    return L, table, n_blocks


@pytest.mark.parametrize("T,cuts,bt", [(700, [0, 256, 640], 16), (512, [0, 128, 384], 32),
                                       (129, [0, 128], 8), (300, [0], 64)])
def test_objects_round_trip_to_the_sequence_encode(T, cuts, bt):
    Hkv = 2
    k, v = _sequence(T, Hkv, seed=T + bt)
    L, table, n_blocks = _paged_pool(T, Hkv, bt, max_tokens=T + 40, seed=T)
    # direct: the whole sequence encoded into the pool
    ref_planes, ref_meta = oracle.encode_batch(L, [T], table, [k], [v], n_blocks)
    # objects serialized, then delivered in shuffled order
    bounds = list(cuts) + [T]
    objs = [(bounds[i], bounds[i + 1] - bounds[i]) for i in range(len(cuts))]
    nbytes = oracle.plane_bytes(L, n_blocks, 64)
    planes = {name: np.zeros(nbytes, np.uint8) for name in ("k_anc", "v_anc", "k_res", "v_res")}
    meta = oracle.Meta.empty(L, 1)
    bufs = {}
    for t0, n in objs:
        bufs[t0] = oracle.serialize(Hkv, n, k[t0:t0 + n], v[t0:t0 + n])
    for t0, n in reversed(objs):
        oracle.deserialize_anchor(L, 0, t0, n, table, bufs[t0][0], planes, meta)
    for name in ("k_anc", "v_anc"):
        assert np.array_equal(planes[name], ref_planes[name]), name
    for name in ("k_scale", "k_zero", "v_scale", "v_zero"):
        assert np.array_equal(getattr(meta, name), getattr(ref_meta, name)), name
    # residual phase: the code planes the merge of the direct planes gives
    codes = {name: np.zeros(2 * nbytes, np.uint8) for name in ("k_codes", "v_codes")}
    for t0, n in objs:
        oracle.deserialize_residual(L, 0, t0, n, table, bufs[t0][1], planes, codes)
    rows = oracle.token_rows(L, table, 0, 0, T).reshape(-1)
    for p, name in (("k", "k_codes"), ("v", "v_codes")):
        full = oracle.merge(ref_planes[p + "_anc"], ref_planes[p + "_res"])
        idx = (rows * 128)[:, None] + np.arange(128)
        assert np.array_equal(codes[name][idx], full[idx]), name
        # rows of no token stay untouched
        mask = np.ones(codes[name].size, bool)
        mask[idx.reshape(-1)] = False
        assert not codes[name][mask].any()


def test_residual_buffer_is_the_residual_planes():
    T, Hkv = 256, 3
    k, v = _sequence(T, Hkv, seed=3)
    anc, res = oracle.serialize(Hkv, T, k, v)
    L = oracle.Layout(Hkv=Hkv, bt=T, max_blocks=1, max_tokens=T)
    planes, _ = oracle.encode_batch(L, [T], np.zeros((1, 1), np.int32), [k], [v], 1)
    s = oracle.serialized_sections(Hkv, T)
    assert np.array_equal(res[: s["k_res"][1]], planes["k_res"])
    assert np.array_equal(res[s["v_res"][0]:], planes["v_res"])
    assert np.array_equal(anc[: s["k_anc"][1]], planes["k_anc"])


def test_object_start_must_be_group_aligned():
    Hkv = 1
    k, v = _sequence(200, Hkv, seed=1)
    L = oracle.Layout(Hkv=Hkv, bt=200, max_blocks=1, max_tokens=200)
    anc, _ = oracle.serialize(Hkv, 100, k[64:164], v[64:164])
    planes = {name: np.zeros(oracle.plane_bytes(L, 1, 64), np.uint8) for name in ("k_anc", "v_anc")}
    with pytest.raises(AssertionError):
        oracle.deserialize_anchor(L, 0, 64, 100, np.zeros((1, 1), np.int32), anc, planes,
                                  oracle.Meta.empty(L, 1))
