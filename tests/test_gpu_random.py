"""Seeded random batches across every supported shape and dtype set, each
compared row for row with the oracle after a KV append (through the C ABI):
random request counts, chunk and context lengths (block and 64-key tile
boundaries included), group sizes, head dims and decode splits."""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import synth  # noqa: E402
from oracle import attention as oa  # noqa: E402
from oracle import kvappend  # noqa: E402
from synth.attn_inputs import make_batch_from_lengths  # noqa: E402
from tests.gpu_util import compare, say  # noqa: E402

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

SHAPES = [  # (H_q, H_kv, D, q/kv dtype)
    (4, 4, 64, "f32"), (8, 2, 128, "f32"), (16, 8, 64, "bf16"), (32, 8, 128, "bf16"),
    (16, 2, 64, "bf16"), (64, 8, 128, "bf16"), (32, 8, 128, "fp8"), (64, 8, 128, "fp8"),
]


def _random_lengths(rng, n_req):
    q, c = [], []
    for _ in range(n_req):
        kind = rng.integers(0, 4)
        if kind == 0:                                   # decode
            qq = 1
        elif kind == 1:                                 # short chunk
            qq = int(rng.integers(2, 40))
        else:                                           # chunk near tile sizes
            qq = int(rng.choice([63, 64, 65, 127, 128, 129, 200]))
        prior = int(rng.choice([0, 1, 15, 16, 17, 63, 64, 65, int(rng.integers(0, 3000))]))
        q.append(qq)
        c.append(qq + prior)
    return q, c


def _wide_lengths(rng, n_req):
    """Longer chunks (up to 512 rows, at and around the planner's tile and
    chunk sizes) and long decodes (up to 12k keys, several split spans)."""
    q, c = [], []
    for _ in range(n_req):
        kind = rng.integers(0, 3)
        if kind == 0:
            qq, prior = 1, int(rng.choice([int(rng.integers(0, 12000)), 4095, 4096, 8191]))
        elif kind == 1:
            qq = int(rng.choice([255, 256, 257, 383, 511, 512]))
            prior = int(rng.choice([0, 16, 1023, int(rng.integers(0, 2500))]))
        else:
            qq = int(rng.integers(2, 130))
            prior = int(rng.integers(0, 6000))
        q.append(qq)
        c.append(qq + prior)
    return q, c


@pytest.mark.parametrize("case", range(24))
def test_random_batch_after_append(case):
    _check_random_case(case, 1000 + case, _random_lengths, [0, 16, 64, 512])


@pytest.mark.parametrize("case", range(40))
def test_wide_random_batch_after_append(case):
    _check_random_case(case, 5000 + case, _wide_lengths, [0, 0, 256, 1024, 3000])


def _check_random_case(case, seed, lengths, splits):
    from paper_2512_04013_amd import runtime as rt
    rng = np.random.default_rng(seed)
    hq, hkv, d, kv = SHAPES[case % len(SHAPES)]
    qd = "f32" if kv == "f32" else "bf16"
    q_lens, ctx_lens = lengths(rng, int(rng.integers(1, 9)))
    split = int(rng.choice(splits))
    sharp = bool(rng.integers(0, 2))
    say(f"[random] seed={seed} case={case} heads={hq}/{hkv} d={d} kv={kv} q={q_lens} ctx={ctx_lens} split={split} sharp={sharp}")
    pool = int(sum(-(-c // 16) for c in ctx_lens)) + 32
    b = make_batch_from_lengths("random", q_lens, ctx_lens, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                                q_dtype=qd, kv_dtype=kv, out_dtype=qd, n_pool_blocks=pool, seed=case,
                                kv_std=1.0 if sharp else 1.0 / np.sqrt(d))
    b = synth.poison_new_slots(b)
    k_new, v_new = synth.make_new_kv(b, seed=case + 7, std=1.0 if sharp else 1.0 / np.sqrt(d))
    shape, kvp, q, bids = rt.upload_batch(b, staging_bytes=1)
    att = rt.MixedAttention(shape, kvp, b.q_start, b.ctx_len, b.bt_start, b.block_ids, bids, kv_split_tokens=split)
    nd = "f32" if kv == "f32" else "bf16"
    att.append(rt.to_device_array(k_new, nd, "cuda"), rt.to_device_array(v_new, nd, "cuda"))
    got = rt.to_host_f64(att.run(q))
    torch.cuda.synchronize()
    k, v, ks, vs = kvappend.append(b.k_cache, b.v_cache, b.k_scale, b.v_scale, kv, k_new, v_new, b.q_start,
                                   b.ctx_len, b.bt_start, b.block_ids)
    assert np.array_equal(kvp.k_cache.contiguous().view(torch.uint8).cpu().numpy().reshape(-1),
                          np.ascontiguousarray(k).view(np.uint8).reshape(-1))
    want = oa.attention_for(b, k_cache=k, v_cache=v, k_scale=ks, v_scale=vs)
    compare(got, want, qd, what=f"random seed {seed} items={att.info.num_items} tiles={att.info.num_prefill_items} "
                                f"groups={att.info.num_merge_groups} row path {att.info.row_path}")
    import paper_2512_04013_amd as aug
    other = None
    if att.info.row_path == aug.AUG_ROWS_MFMA:
        other = aug.AUG_ROWS_VALU          # eight-head groups: also the vector-ALU rows
    elif hq == 4 * hkv and d == 128 and qd == "bf16":
        other = aug.AUG_ROWS_MFMA          # four-head groups: also the opt-in MFMA rows
    if other is not None:
        att2 = rt.MixedAttention(shape, kvp, b.q_start, b.ctx_len, b.bt_start, b.block_ids, bids,
                                 kv_split_tokens=split, row_path=other)
        assert att2.info.row_path == other
        got2 = rt.to_host_f64(att2.run(q))
        torch.cuda.synchronize()
        compare(got2, want, qd, what=f"random seed {seed} row path {other}")
