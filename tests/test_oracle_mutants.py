"""The pins are strong enough: plausible mistakes planted in the oracle (on
the CPU, one at a time) each make at least one pin fail.

Every mutant replaces one oracle function with a copy that has a single
planted error (an off-by-one, a wrong index map, a dropped term, a swapped
operand, a wrong comparison), then runs the pin tests of that part of the
oracle and counts how many fail."""

import inspect

import numpy as np
import pytest

from oracle import attention as oa
from oracle import former as of
from oracle import kvappend as ka
from oracle import kvpark as kp
from oracle import codecs as oc
from oracle.codecs import E4M3FN_TABLE, bf16_bits_to_f64, e4m3fn_encode
from tests import test_oracle_append as pins_append
from tests import test_oracle_attention as pins_attention
from tests import test_oracle_former as pins_former


def _run_pins(module, stop_at_first=True):
    """Run every test function of ``module`` (parametrized ones on their
    parameter sets) until one fails (or all, without ``stop_at_first``);
    returns (failures, runs)."""
    fails = runs = 0
    for name, fn in inspect.getmembers(module, inspect.isfunction):
        if not name.startswith("test_") or fn.__module__ != module.__name__:
            continue
        marks = getattr(fn, "pytestmark", [])
        params = [m for m in marks if m.name == "parametrize"]
        if any(m.name == "skipif" and m.args and m.args[0] for m in marks):
            continue
        cases = [{}]
        for m in params:
            argnames = [a.strip() for a in m.args[0].split(",")] if isinstance(m.args[0], str) else list(m.args[0])
            new = []
            for c in cases:
                for v in m.args[1]:
                    vals = v if len(argnames) > 1 else (v,)
                    new.append({**c, **dict(zip(argnames, vals))})
            cases = new
        for kw in cases:
            runs += 1
            try:
                fn(**kw)
            except Exception:   # an assertion, or a mutant crashing a pin: both are catches
                fails += 1
                if stop_at_first:
                    return fails, runs
    return fails, runs


# ---- attention ---------------------------------------------------------------------------

def _attend(offset=0, gqa_mod=False, scale=True, swap_kv=False, causal=True):
    def attend(q_rows, k, v, num_q_heads, num_kv_heads, softmax_scale):
        q_len, ctx = q_rows.shape[0], k.shape[0]
        group = num_q_heads // num_kv_heads
        pos = ctx - q_len + np.arange(q_len) + offset
        masked = np.arange(ctx)[None, :] > pos[:, None]
        out = np.empty_like(q_rows)
        for h in range(num_q_heads):
            g = h % num_kv_heads if gqa_mod else h // group
            s = q_rows[:, h, :] @ k[:, g, :].T
            if scale:
                s = s * softmax_scale
            if causal:
                s[masked] = -np.inf
            s -= s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            out[:, h, :] = p @ (k[:, g, :] if swap_kv else v[:, g, :])
        return out
    return attend


def _materialise(reverse=False, no_scale=False):
    def materialise(cache, scale, kv_dtype, blocks, ctx):
        nblk = -(-ctx // oa.BLOCK)
        blocks = np.asarray(blocks[:nblk], dtype=np.int64)
        if reverse:
            blocks = blocks[::-1]
        raw = oa.storage_to_f64(cache[blocks], kv_dtype)
        if kv_dtype == "fp8" and not no_scale:
            raw = raw * scale[blocks].astype(np.float64)[:, :, None, None]
        h_kv, d = raw.shape[1], raw.shape[3]
        return raw.transpose(0, 2, 1, 3).reshape(nblk * oa.BLOCK, h_kv, d)[:ctx]
    return materialise


ATTENTION_MUTANTS = {
    "causal position one too early": ("attend_request", _attend(offset=-1)),
    "causal position one too late": ("attend_request", _attend(offset=+1)),
    "GQA head map h % H_kv": ("attend_request", _attend(gqa_mod=True)),
    "softmax scale dropped": ("attend_request", _attend(scale=False)),
    "K used in place of V": ("attend_request", _attend(swap_kv=True)),
    "no causal mask": ("attend_request", _attend(causal=False)),
    "block table walked backwards": ("materialise_kv", _materialise(reverse=True)),
    "fp8 block scale ignored": ("materialise_kv", _materialise(no_scale=True)),
}


@pytest.mark.parametrize("mutant", sorted(ATTENTION_MUTANTS))
def test_attention_pins_catch(mutant, monkeypatch):
    name, fn = ATTENTION_MUTANTS[mutant]
    monkeypatch.setattr(oa, name, fn)
    fails, runs = _run_pins(pins_attention)
    assert fails > 0, f"{mutant}: none of {runs} attention pins failed"


# ---- KV append ---------------------------------------------------------------------------

def _segments(slot_shift=0):
    def segments(q_start, ctx_len, bt_start):
        out = []
        for r in range(len(ctx_len)):
            q = int(q_start[r + 1] - q_start[r])
            first = int(ctx_len[r]) - q + slot_shift
            p = first
            while p < int(ctx_len[r]) + slot_shift:
                blk = p // ka.BLOCK
                end = min(int(ctx_len[r]) + slot_shift, (blk + 1) * ka.BLOCK)
                out.append((r, blk, int(q_start[r]) + p - first, end - p, p % ka.BLOCK))
                p = end
        return out
    return segments


def _append_fp8(no_reencode=False, always_new=False, keep_old=False):
    def append_fp8(cache, scale, new_bits, segs, bt_start, block_ids, h_kv):
        for r, blk, row0, n, slot0 in segs:
            b = int(block_ids[int(bt_start[r]) + blk])
            for h in range(h_kv):
                x = bf16_bits_to_f64(new_bits[row0:row0 + n, h, :]).astype(np.float32)
                need = np.float32(np.float32(np.abs(x).max()) / ka.FP8_MAX)
                s_old = np.float32(scale[b, h])
                if slot0 == 0 or always_new:
                    s = need
                elif keep_old:
                    s = s_old
                else:
                    s = need if need > s_old else s_old
                    if s > s_old and not no_reencode:
                        old = E4M3FN_TABLE[cache[b, h, :slot0, :]].astype(np.float32)
                        cache[b, h, :slot0, :] = e4m3fn_encode(np.float32(old * s_old) / s)
                codes = np.zeros(x.shape, np.uint8) if s == 0 else e4m3fn_encode(x / s)
                cache[b, h, slot0:slot0 + n, :] = codes
                scale[b, h] = s
    return append_fp8


APPEND_MUTANTS = {
    "new rows one slot late": ("append_segments", _segments(slot_shift=1)),
    "earlier codes not re-encoded when the scale grows": ("_append_fp8", _append_fp8(no_reencode=True)),
    "scale always from the new rows": ("_append_fp8", _append_fp8(always_new=True)),
    "scale never grows": ("_append_fp8", _append_fp8(keep_old=True)),
}


@pytest.mark.parametrize("mutant", sorted(APPEND_MUTANTS))
def test_append_pins_catch(mutant, monkeypatch):
    name, fn = APPEND_MUTANTS[mutant]
    monkeypatch.setattr(ka, name, fn)
    fails, runs = _run_pins(pins_append)
    assert fails > 0, f"{mutant}: none of {runs} append pins failed"


# ---- number formats ----------------------------------------------------------------------

def _e4m3(bias=7, subnormal_as_normal=False, nan_only_all_ones=False):
    def value(code):
        code = int(code) & 0xFF
        sign = -1.0 if code & 0x80 else 1.0
        e, m = (code >> 3) & 0xF, code & 0x7
        if (code & 0x7F) == 0x7F and not nan_only_all_ones or code == 0xFF and nan_only_all_ones:
            return float("nan")
        if e == 0 and not subnormal_as_normal:
            return sign * m * 2.0 ** -9
        return sign * (1.0 + m / 8.0) * 2.0 ** (e - bias)
    return value


FORMAT_MUTANTS = {
    "E4M3FN exponent bias 8": _e4m3(bias=8),
    "E4M3FN subnormals read as normals": _e4m3(subnormal_as_normal=True),
    "E4M3FN NaN only at 0xFF": _e4m3(nan_only_all_ones=True),
}


@pytest.mark.parametrize("mutant", sorted(FORMAT_MUTANTS))
def test_format_pins_catch(mutant, monkeypatch):
    fn = FORMAT_MUTANTS[mutant]
    monkeypatch.setattr(oc, "e4m3fn_value", fn)
    monkeypatch.setattr(oc, "E4M3FN_TABLE", np.array([fn(c) for c in range(256)], dtype=np.float64))
    fails, runs = _run_pins(pins_attention)
    assert fails > 0, f"{mutant}: none of {runs} attention pins failed"


def test_bf16_decoder_mutant_is_caught(monkeypatch):
    def shifted(u16):   # bf16 bits placed one position too low in the float32
        u32 = np.asarray(u16, dtype=np.uint16).astype(np.uint32) << np.uint32(15)
        return u32.view(np.float32).astype(np.float64)
    monkeypatch.setattr(oc, "bf16_bits_to_f64", shifted)
    fails, runs = _run_pins(pins_attention)
    assert fails > 0, f"bf16 decoder shifted: none of {runs} attention pins failed"


# ---- park / resume -----------------------------------------------------------------------

def _park(v_first=False, no_scales=False, k_scale_twice=False, sort_blocks=False):
    def park(k_cache, v_cache, k_scale, v_scale, kv_dtype, blocks):
        parts = []
        blocks = np.asarray(blocks, dtype=np.int64)
        for b in (np.sort(blocks) if sort_blocks else blocks):
            kb = np.ascontiguousarray(k_cache[b]).view(np.uint8).ravel()
            vb = np.ascontiguousarray(v_cache[b]).view(np.uint8).ravel()
            parts += [vb, kb] if v_first else [kb, vb]
            if kv_dtype == "fp8" and not no_scales:
                parts.append(np.ascontiguousarray(k_scale[b], dtype=np.float32).view(np.uint8).ravel())
                second = k_scale if k_scale_twice else v_scale
                parts.append(np.ascontiguousarray(second[b], dtype=np.float32).view(np.uint8).ravel())
        return np.concatenate(parts) if parts else np.zeros(0, np.uint8)
    return park


def _resume_reversed(k_cache, v_cache, k_scale, v_scale, kv_dtype, blocks, image):
    return _ORIGINAL_RESUME(k_cache, v_cache, k_scale, v_scale, kv_dtype, np.asarray(blocks)[::-1], image)


_ORIGINAL_RESUME = kp.resume

PARK_MUTANTS = {
    "V before K in a record": ("park", _park(v_first=True)),
    "fp8 scales left out of the record": ("park", _park(no_scales=True)),
    "K scale written in place of the V scale": ("park", _park(k_scale_twice=True)),
    "blocks parked in sorted order, not the listed one": ("park", _park(sort_blocks=True)),
    "records resumed into the blocks in reverse": ("resume", _resume_reversed),
}


@pytest.mark.parametrize("mutant", sorted(PARK_MUTANTS))
def test_park_pins_catch(mutant, monkeypatch):
    name, fn = PARK_MUTANTS[mutant]
    monkeypatch.setattr(kp, name, fn)
    fails, runs = _run_pins(pins_attention)
    assert fails > 0, f"{mutant}: none of {runs} attention and park pins failed"


# ---- batch former ------------------------------------------------------------------------

FORMER_MUTANTS = {
    "priority inverted (C / V)": ("priority", lambda p, c, w_ms: c / (1.0 + p.beta * w_ms)),
    "aging term dropped": ("priority", lambda p, c, w_ms: 1.0 / c),
    "budget not clipped": ("token_budget",
                           lambda p, free, pre, bs: (free + pre) * bs),
    "budget counts free blocks only": ("token_budget",
                                       lambda p, free, pre, bs: min(max(free * bs, int(np.floor(p.beta_low * p.t_max))),
                                                                    int(np.floor(p.beta_high * p.t_max)))),
    "prefill chunk not capped": ("tokens_of", lambda p, r, budget: r.pending if r.pending > 0 else 1),
    "decode cost missing the triangle term": ("decode_cost", lambda p, l0, n: float(n * l0) * p.t_iter),
    "Waste ties to Swap first": ("select_policy",
                                 lambda p, lt, tau, lo: [of.SWAP, of.DISCARD, of.PRESERVE][
                                     int(np.argmin(list(of.waste(p, lt, tau, lo))[::-1]))]),
}


@pytest.mark.parametrize("mutant", sorted(FORMER_MUTANTS))
def test_former_pins_catch(mutant, monkeypatch):
    name, fn = FORMER_MUTANTS[mutant]
    monkeypatch.setattr(of, name, fn)
    fails, runs = _run_pins(pins_former)
    assert fails > 0, f"{mutant}: none of {runs} former pins failed"


def test_unmutated_oracle_passes_every_pin():
    for module in (pins_attention, pins_append, pins_former):
        fails, runs = _run_pins(module, stop_at_first=False)
        assert runs > 5 and fails == 0, (module.__name__, fails, runs)
