"""GPU parity of aug_kv_append against the oracle (through the C ABI): the
pool and the fp8 scales bit-exact after the append, and the same step's
attention over the appended cache within the attention tolerances."""

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


def _bytes(t):
    return t.contiguous().view(torch.uint8).cpu().numpy().reshape(-1)


def _same(got, want, what):
    """Byte equality, reported as a count of differing bytes (never the arrays)."""
    want = np.ascontiguousarray(want).view(np.uint8).reshape(-1)
    assert got.size == want.size, f"{what}: {got.size} bytes vs {want.size}"
    bad = np.count_nonzero(got != want)
    assert bad == 0, f"{what}: {bad} of {got.size} bytes differ (first at {int(np.argmax(got != want))})"


def _new_rows_to_device(k_new, v_new, kv):
    from paper_2512_04013_amd import runtime as rt
    dt = "f32" if kv == "f32" else "bf16"
    return rt.to_device_array(k_new, dt, "cuda"), rt.to_device_array(v_new, dt, "cuda")


def _append_on_gpu(b, k_new, v_new):
    from paper_2512_04013_amd import runtime as rt
    shape, kv, q, bids = rt.upload_batch(b)
    att = rt.MixedAttention(shape, kv, b.q_start, b.ctx_len, b.bt_start, b.block_ids, bids)
    kd, vd = _new_rows_to_device(k_new, v_new, b.kv_dtype)
    att.append(kd, vd)
    return att, kv, q


CASES = [
    # (q_lens, ctx_lens, hq, hkv, d, kv dtype, std of the new rows)
    ([20, 1, 1, 33, 1, 7], [25, 17, 16, 70, 1, 7], 4, 4, 64, "f32", 1.0),
    ([1, 70, 1, 3, 128], [200, 70, 1000, 29, 700], 8, 4, 128, "f32", 1.0),
    ([33, 1, 129, 1, 16], [100, 1, 500, 2049, 48], 32, 8, 128, "bf16", 1.0),
    ([1, 9, 1, 40], [513, 100, 48, 41], 16, 4, 64, "bf16", 1.0),
    ([130, 1, 64, 17, 1, 1], [1500, 700, 64, 3000, 32, 40], 64, 8, 128, "fp8", 1.0),
    ([130, 1, 64, 17, 1, 1], [1500, 700, 64, 3000, 32, 40], 64, 8, 128, "fp8", 6.0),    # scales grow
    ([130, 1, 64, 17, 1, 1], [1500, 700, 64, 3000, 32, 40], 64, 8, 128, "fp8", 0.05),   # scales kept
    ([3, 1, 2], [19, 9, 2], 16, 2, 128, "fp8", 0.0),                                     # zero rows
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_append_is_bit_exact_and_attention_reads_it(case):
    q_lens, ctx_lens, hq, hkv, d, kv, std = CASES[case]
    qd = "f32" if kv == "f32" else "bf16"
    say(f"[append] case={case} kv={kv} q={q_lens} ctx={ctx_lens} heads={hq}/{hkv} d={d} std={std}")
    b = make_batch_from_lengths("append", q_lens, ctx_lens, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                                q_dtype=qd, kv_dtype=kv, out_dtype=qd, n_pool_blocks=640, seed=case)
    b = synth.poison_new_slots(b)
    k_new, v_new = synth.make_new_kv(b, seed=50 + case, std=std)
    att, kvp, q = _append_on_gpu(b, k_new, v_new)
    torch.cuda.synchronize()
    k, v, ks, vs = kvappend.append(b.k_cache, b.v_cache, b.k_scale, b.v_scale, kv, k_new, v_new,
                                   b.q_start, b.ctx_len, b.bt_start, b.block_ids)
    _same(_bytes(kvp.k_cache), np.ascontiguousarray(k).view(np.uint8).reshape(-1), "kvp.k_cache")
    _same(_bytes(kvp.v_cache), np.ascontiguousarray(v).view(np.uint8).reshape(-1), "kvp.v_cache")
    if kv == "fp8":
        _same(_bytes(kvp.k_scale), ks.view(np.uint8).reshape(-1), "kvp.k_scale")
        _same(_bytes(kvp.v_scale), vs.view(np.uint8).reshape(-1), "kvp.v_scale")
    out = att.run(q)
    torch.cuda.synchronize()
    from paper_2512_04013_amd import runtime as rt
    want = oa.attention_for(b, k_cache=k, v_cache=v, k_scale=ks, v_scale=vs)
    got = rt.to_host_f64(out)
    if std <= 1.0:
        compare(got, want, qd, what=f"attention after append, case {case}")
        return
    # New rows far larger than the configured N(0,1) inputs. A departure from
    # the stated gate, on purpose: the bf16 and fp8 paths round each probability to
    # bf16 (relative 2^-9) before the P.V product, which moves an output by at
    # most 2^-9 * max|v - o| / (1 - 2^-9) <= 2^-8 * max|v|, plus half an ulp
    # of the bf16 output; the fixed 1e-2 gate therefore holds only while
    # max|v| stays within a few units (it does for every configured workload,
    # sharp inputs included), and this case is held to that derived bound.
    vmax = max(np.abs(oa.materialise_kv(v, vs, kv, b.blocks_of(r), int(b.ctx_len[r]))).max()
               for r in range(b.num_reqs))
    bound = 2.0 ** -8 * vmax + 2.0 ** -9 * np.abs(want) + 1e-6
    worst = float((np.abs(got - want) / bound).max())
    rel = float((np.sqrt(((got - want) ** 2).sum(-1)) / np.sqrt((want ** 2).sum(-1))).max())
    say(f"  case {case}: max|v|={vmax:.2f}, worst error / bound = {worst:.3f}, rel_l2={rel:.3e}")
    assert worst <= 1.0 and rel <= 2e-2


def test_append_twice_into_the_same_blocks_follows_the_oracle():
    # two consecutive decode steps of fp8 requests: the second appends into
    # the blocks (and scales) the first one wrote, or opens a new block
    from paper_2512_04013_amd import runtime as rt
    c = np.array([16, 31, 63, 99], np.int32)          # step 0 writes position c - 1, step 1 position c
    b1 = make_batch_from_lengths("append2", [1] * 4, c + 1, num_q_heads=64, num_kv_heads=8, head_dim=128,
                                 q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16", n_pool_blocks=64, seed=3)
    b1 = synth.poison_new_slots(b1)
    say("[append] two decode steps into shared fp8 blocks")
    shape, kvp, _, bids = rt.upload_batch(b1)
    k, v, ks, vs = b1.k_cache, b1.v_cache, b1.k_scale, b1.v_scale
    qs = np.arange(5, dtype=np.int32)
    for step in range(2):
        ctx = c + step
        k_new, v_new = synth.make_new_kv(b1, seed=70 + step, std=1.0 + 3.0 * step)
        att = rt.MixedAttention(shape, kvp, qs, ctx, b1.bt_start, b1.block_ids, bids)
        kd, vd = _new_rows_to_device(k_new, v_new, "fp8")
        att.append(kd, vd)
        k, v, ks, vs = kvappend.append(k, v, ks, vs, "fp8", k_new, v_new, qs, ctx, b1.bt_start, b1.block_ids)
        torch.cuda.synchronize()
    _same(_bytes(kvp.k_cache), k.reshape(-1), "kvp.k_cache")
    _same(_bytes(kvp.v_cache), v.reshape(-1), "kvp.v_cache")
    _same(_bytes(kvp.k_scale), ks.view(np.uint8).reshape(-1), "kvp.k_scale")
    _same(_bytes(kvp.v_scale), vs.view(np.uint8).reshape(-1), "kvp.v_scale")


def _touched_blocks(b):
    segs = kvappend.append_segments(b.q_start, b.ctx_len, b.bt_start)
    return np.array(sorted({int(b.block_ids[int(b.bt_start[r]) + blk]) for r, blk, *_ in segs}), np.int64)


def _oracle_on_touched(b, k_new, v_new, touched):
    """The oracle's append run on a sub-pool holding only the touched blocks
    (every other table entry points past the sub-pool, so a stray access fails)."""
    remap = np.full(b.num_pool_blocks, len(touched), np.int64)
    remap[touched] = np.arange(len(touched))
    sub_ids = remap[b.block_ids]
    sk = None if b.k_scale is None else b.k_scale[touched]
    sv = None if b.v_scale is None else b.v_scale[touched]
    return kvappend.append(b.k_cache[touched], b.v_cache[touched], sk, sv, b.kv_dtype, k_new, v_new,
                           b.q_start, b.ctx_len, b.bt_start, sub_ids)


@pytest.mark.parametrize("which", ["mixed-8b-bf16", "prefill-heavy-fp8"])
def test_append_full_size(which):
    from paper_2512_04013_amd import runtime as rt
    if which == "mixed-8b-bf16":
        b = synth.make_mixed_8b(seed=0)
        # the resumed requests' KV as after their resume (park and resume have tests of their own)
        b.k_cache[b.park.resume_blocks] = b.k_cache[b.park.resume_src_blocks]
        b.v_cache[b.park.resume_blocks] = b.v_cache[b.park.resume_src_blocks]
        b.park = None
    else:
        rng = np.random.default_rng(7)
        q_lens = [512] * 14 + [1] * 512
        ctx_lens = [512 + int(x) for x in rng.integers(0, 3000, 14)] + \
            [int(x) for x in np.clip(rng.lognormal(np.log(2500), 0.8, 512), 1, 16384)]
        b = make_batch_from_lengths("prefill-heavy-fp8", q_lens, ctx_lens, num_q_heads=64, num_kv_heads=8,
                                    head_dim=128, q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16",
                                    n_pool_blocks=160_000, seed=8)
    synth.poison_new_slots(b, copy=False)
    say(f"[append full] {which}: {b.num_reqs} requests, {b.total_q} rows")
    k_new, v_new = synth.make_new_kv(b, seed=11, std=1.0 / np.sqrt(128.0))
    att, kvp, q = _append_on_gpu(b, k_new, v_new)
    out = att.run(q)
    torch.cuda.synchronize()
    touched = _touched_blocks(b)
    assert len(touched) == att.info.num_append_items
    k, v, ks, vs = _oracle_on_touched(b, k_new, v_new, touched)
    tt = torch.from_numpy(touched).cuda()
    _same(_bytes(kvp.k_cache[tt]), np.ascontiguousarray(k).view(np.uint8).reshape(-1), "kvp.k_cache[tt]")
    _same(_bytes(kvp.v_cache[tt]), np.ascontiguousarray(v).view(np.uint8).reshape(-1), "kvp.v_cache[tt]")
    if b.kv_dtype == "fp8":
        _same(_bytes(kvp.k_scale[tt]), ks.view(np.uint8).reshape(-1), "kvp.k_scale[tt]")
        _same(_bytes(kvp.v_scale[tt]), vs.view(np.uint8).reshape(-1), "kvp.v_scale[tt]")
    # a sample of the other blocks is untouched
    others = np.setdiff1d(np.random.default_rng(1).choice(b.num_pool_blocks, 4000, replace=False), touched)
    ot = torch.from_numpy(others).cuda()
    _same(_bytes(kvp.k_cache[ot]), np.ascontiguousarray(b.k_cache[others]).view(np.uint8).reshape(-1), "kvp.k_cache[ot]")
    # attention of every row over the appended cache
    b.k_cache[touched], b.v_cache[touched] = k, v
    if b.kv_dtype == "fp8":
        b.k_scale[touched], b.v_scale[touched] = ks, vs
    want = oa.attention_for(b)
    compare(rt.to_host_f64(out), want, "bf16", what=f"{which} after append (all {b.total_q} rows)")
