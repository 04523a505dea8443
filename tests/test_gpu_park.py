"""GPU tests of aug_kv_park / aug_kv_resume: bit-exact against the oracle's
byte image, for every KV dtype and with staging smaller than the image."""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import kvpark  # noqa: E402
from synth.attn_inputs import make_batch_from_lengths  # noqa: E402
from tests.gpu_util import say  # noqa: E402
import synth  # noqa: E402

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


@pytest.mark.parametrize("kv", ["f32", "bf16", "fp8"])
@pytest.mark.parametrize("staging_records", [1, 3, 1000])
def test_park_resume_roundtrip_is_bit_exact(kv, staging_records):
    from paper_2512_04013_amd import runtime as rt
    qd = "f32" if kv == "f32" else "bf16"
    hq, hkv, d = (8, 8, 64) if kv == "f32" else (64, 8, 128)
    b = make_batch_from_lengths("park", [1, 1], [100, 37], num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                                q_dtype=qd, kv_dtype=kv, out_dtype=qd, n_pool_blocks=64, seed=11,
                                extra_reqs_ctx=[90, 33])
    say(f"[park] kv={kv} staging_records={staging_records}")
    shape, pool, q, bids = rt.upload_batch(b, staging_bytes=1)
    pool.staging = torch.empty(staging_records * pool.record_bytes, dtype=torch.uint8, device="cuda")
    src = b.park.park_blocks
    used = set(b.block_ids.tolist()) | set(src.tolist())
    dst = np.array(sorted(set(range(64)) - used)[:len(src)], np.int32)
    host = pool.host_buffer(len(src))
    pool.park(src, torch.from_numpy(src).cuda(), host)
    torch.cuda.synchronize()
    want = kvpark.park(b.k_cache, b.v_cache, b.k_scale, b.v_scale, kv, src)
    assert host.numpy().size == want.size and np.array_equal(host.numpy(), want)
    before_k = pool.k_cache.view(torch.uint8).cpu().numpy().copy()
    pool.resume(dst, torch.from_numpy(dst).cuda(), host)
    torch.cuda.synchronize()
    k2, v2, ks2, vs2 = kvpark.resume(b.k_cache, b.v_cache, b.k_scale, b.v_scale, kv, dst, want)
    got_k = pool.k_cache.view(torch.uint8).cpu().numpy()
    got_v = pool.v_cache.view(torch.uint8).cpu().numpy()
    assert np.array_equal(got_k, np.ascontiguousarray(k2).view(np.uint8).reshape(got_k.shape))
    assert np.array_equal(got_v, np.ascontiguousarray(v2).view(np.uint8).reshape(got_v.shape))
    if kv == "fp8":
        assert np.array_equal(pool.k_scale.cpu().numpy().view(np.uint32), ks2.view(np.uint32))
        assert np.array_equal(pool.v_scale.cpu().numpy().view(np.uint32), vs2.view(np.uint32))
    others = np.setdiff1d(np.arange(64), dst)
    assert np.array_equal(got_k.reshape(64, -1)[others], before_k.reshape(64, -1)[others])


def test_tiny_mixed_paused_request_round_trip():
    from paper_2512_04013_amd import runtime as rt
    b = synth.make_tiny_mixed(seed=4)
    say("[park] tiny mixed paused request")
    shape, pool, q, bids = rt.upload_batch(b)
    pk = b.park
    host = pool.host_buffer(len(pk.park_blocks))
    pool.park(pk.park_blocks, torch.from_numpy(pk.park_blocks).cuda(), host)
    pool.resume(pk.resume_blocks, torch.from_numpy(pk.resume_blocks).cuda(), host)
    torch.cuda.synchronize()
    k = pool.k_cache.cpu().numpy()
    assert np.array_equal(k[pk.resume_blocks].view(np.uint32), b.k_cache[pk.park_blocks].view(np.uint32))
    v = pool.v_cache.cpu().numpy()
    assert np.array_equal(v[pk.resume_blocks].view(np.uint32), b.v_cache[pk.park_blocks].view(np.uint32))
