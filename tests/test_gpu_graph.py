"""The plan upload and several layers of one planned batch (KV append, then
attention, per layer, each layer with its own pool, block table, queries and
new rows) captured in a HIP graph: every replay reproduces the eager launches bit for bit, with the
program's own eager work and synchronisations between replays."""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2512_04013_amd as aug  # noqa: E402
import synth  # noqa: E402
from oracle import attention as oa  # noqa: E402
from oracle import kvappend  # noqa: E402
from synth.attn_inputs import make_batch_from_lengths  # noqa: E402
from tests.gpu_util import compare, say  # noqa: E402

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

LAYERS = 4


def _bytes(t):
    return t.contiguous().view(torch.uint8).cpu().numpy().reshape(-1)


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
def test_layers_in_a_graph_replay_the_eager_bits(kv):
    from paper_2512_04013_amd import runtime as rt
    hq = 64 if kv == "fp8" else 32
    # a prefill chunk over prior context (tiles, split along keys), decodes with
    # split spans (merged inside the launch) and short decodes
    q_lens, ctx_lens = [130, 1, 1, 1, 17], [2600, 4100, 900, 33, 17]
    layers = []
    for l in range(LAYERS):
        b = make_batch_from_lengths("graph", q_lens, ctx_lens, num_q_heads=hq, num_kv_heads=8, head_dim=128,
                                    q_dtype="bf16", kv_dtype=kv, out_dtype="bf16", n_pool_blocks=700, seed=40 + l)
        b = synth.poison_new_slots(b)
        k_new, v_new = synth.make_new_kv(b, seed=60 + l)
        shape, pool, q, bids = rt.upload_batch(b, staging_bytes=1)
        layers.append(dict(b=b, pool=pool, q=q, bids=bids, k_new=rt.to_device_array(k_new, "bf16", "cuda"),
                           v_new=rt.to_device_array(v_new, "bf16", "cuda"), k_new_h=k_new, v_new_h=v_new,
                           out=torch.empty((b.total_q, hq, 128), dtype=torch.bfloat16, device="cuda")))
    b0 = layers[0]["b"]
    att = rt.MixedAttention(shape, layers[0]["pool"], b0.q_start, b0.ctx_len, b0.bt_start, b0.block_ids,
                            layers[0]["bids"], kv_split_tokens=512)
    say(f"[graph] kv={kv} {LAYERS} layers, items={att.info.num_items} tiles={att.info.num_prefill_items} "
        f"groups={att.info.num_merge_groups} tile merges={att.info.num_tile_merge_groups}")
    assert att.info.num_merge_groups > att.info.num_tile_merge_groups > 0

    plan_bytes = int(att.info.plan_bytes)

    def one_step(stream=None):
        # the step's plan image from its pinned host copy, then every layer
        aug.aug_plan_upload(att.plan_host, att.plan_dev, plan_bytes, stream=stream)
        for L in layers:
            att.append(L["k_new"], L["v_new"], stream=stream, kv=L["pool"], block_ids=L["bids"])
            att.run(L["q"], stream=stream, kv=L["pool"], block_ids=L["bids"], out=L["out"])

    one_step()
    torch.cuda.synchronize()
    eager = [(_bytes(L["out"]), _bytes(L["pool"].k_cache), _bytes(L["pool"].v_cache)) for L in layers]
    # layer 0 against the oracle, after its append
    L0 = layers[0]
    kk, vv, ks, vs = kvappend.append(b0.k_cache, b0.v_cache, b0.k_scale, b0.v_scale, kv, L0["k_new_h"],
                                     L0["v_new_h"], b0.q_start, b0.ctx_len, b0.bt_start, b0.block_ids)
    want = oa.attention_for(b0, k_cache=kk, v_cache=vv, k_scale=ks, v_scale=vs)
    compare(rt.to_host_f64(L0["out"]), want, "bf16", what=f"graph layer 0 eager ({kv})")

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        one_step()                                   # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        one_step(stream=torch.cuda.current_stream().cuda_stream)
    scratch = torch.empty_like(layers[0]["out"])
    for rep in range(3):
        for L in layers:
            L["out"].zero_()
        # eager work of the program between replays
        att.run(layers[1]["q"], kv=layers[1]["pool"], block_ids=layers[1]["bids"], out=scratch)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for l, L in enumerate(layers):
            got = (_bytes(L["out"]), _bytes(L["pool"].k_cache), _bytes(L["pool"].v_cache))
            for name, x, y in zip(("out", "k", "v"), got, eager[l]):
                assert np.array_equal(x, y), f"replay {rep} layer {l} {name}: {np.count_nonzero(x != y)} bytes differ"
        assert np.array_equal(_bytes(scratch), eager[1][0])
    say(f"  {kv}: 3 replays of {LAYERS} layers identical to the eager launches")
