"""GPU parity of the batched composition at full size, in the launch
configuration bench.py times: 16 sequences each splice three library skills
(1024, 2048, 4096 tokens) at random disjoint offsets into 8k-12k contexts
with one pkv_reposition_splice_batched call, then a 256-query causal suffix
per sequence attends over its own cache with one ragged pkv_suffix_attention
call (paper Sec. 5: a library of skills composes; Sec. 6 delta prefill).

Two layers (first and last) are checked.  For those layers every oracle input
is built on the host from the seeded draws: the skill library rotated to its
source positions, the suffix keys and queries rotated to theirs, and the
pre-splice cache; these are uploaded in place of the device-prepared data
before the timed launches run.  Bars as elsewhere: values bit-exact, keys
within one bf16 ulp, attention max-abs 2e-2 / mean-abs 2e-3 / rel-L2 1e-2 on
sampled rows (three queries per sequence, all heads)."""
import numpy as np
import pytest
import torch

import bench
import oracle
from helpers import bits_to_f64, check_attention_close, check_rotated_keys, dev, host_bits, log
from paper_2606_17107_amd import pkv, synth

pytestmark = pytest.mark.gpu

LAYERS = [0, 31]


def rope_positions(x_pre, positions, theta, d):
    """Oracle RoPE of rows [..., T, d] at per-token positions (fp64, one rounding)."""
    pos = np.broadcast_to(np.asarray(positions, dtype=np.int32), x_pre.shape[:-1]).copy()
    return oracle.rope_rows(np.ascontiguousarray(x_pre), pos, theta, d)


def test_full_batched():
    bw = synth.BATCHED
    torch.cuda.synchronize()
    log("full-size batched: building the bench step")
    step = bench.BatchedStep(bw, 0)
    plan = step.plan
    d, nq = bw.head_dim, bw.n_q
    # The same seeded draws again (device generator, same order) for the checked layers.
    c = synth.batched_case(bw, plan, seed=0, device="cuda")
    host = {k: host_bits(v[LAYERS]) for k, v in c.items()}
    del c
    torch.cuda.empty_cache()

    # Oracle-prepared inputs of the checked layers.
    lib_pos = np.concatenate([np.arange(plan["src_pos0"][k], plan["src_pos0"][k] + n, dtype=np.int32)
                              for k, n in enumerate(bw.skills)])
    skill_k = rope_positions(host["skill_k_pre"], lib_pos, bw.theta, d)
    cache_k, cache_v = host["ctx_k"].copy(), host["ctx_v"].copy()
    q = np.empty_like(host["q_pre"])
    q_pos = np.empty(bw.n_seqs * nq, dtype=np.int32)
    for s_i, sq in enumerate(plan["seqs"]):
        C, base = sq["ctx"], sq["seq_base"]
        rows = slice(s_i * nq, (s_i + 1) * nq)
        pos = np.arange(C, C + nq, dtype=np.int32)
        q_pos[rows] = pos
        cache_k[:, :, base + C: base + C + nq] = rope_positions(host["suf_k_pre"][:, :, rows], pos, bw.theta, d)
        cache_v[:, :, base + C: base + C + nq] = host["suf_v"][:, :, rows]
        qt = np.ascontiguousarray(host["q_pre"][:, rows].transpose(0, 2, 1, 3))   # [L][H][n_q][d]
        q[:, rows] = rope_positions(qt, pos, bw.theta, d).transpose(0, 2, 1, 3)
    for i, l in enumerate(LAYERS):
        step.skill_k[l] = dev(skill_k[i])
        step.cache_k[l] = dev(cache_k[i])
        step.cache_v[l] = dev(cache_v[i])
        step.q[l] = dev(q[i])
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream().cuda_stream
    log("batched splice: %d segments" % len(step.segs))
    step.splice(stream)
    torch.cuda.synchronize()
    got_k = host_bits(step.cache_k[LAYERS])
    got_v = host_bits(step.cache_v[LAYERS])

    # Oracle splice, segment by segment, on each sequence's own slot axis.
    want_k, want_v = cache_k, cache_v
    for sg in step.segs:
        n = sg["n_tokens"]
        src = slice(sg["src_slot0"], sg["src_slot0"] + n)
        base, ln = sg["dst_seq_base"], sg["dst_seq_len"]
        oracle.reposition_splice(np.ascontiguousarray(skill_k[:, :, src]),
                                 np.ascontiguousarray(host["skill_v"][:, :, src]),
                                 want_k[:, :, base: base + ln], want_v[:, :, base: base + ln],
                                 np.arange(sg["src_pos0"], sg["src_pos0"] + n, dtype=np.int32),
                                 np.arange(sg["dst_pos0"], sg["dst_pos0"] + n, dtype=np.int32), bw.theta, d)
    np.testing.assert_array_equal(got_v, want_v)
    n_diff, n_floor = check_rotated_keys(got_k, want_k, 0, d, synth.HALF)
    log("  K elements not bit-equal:", n_diff, "needing the floor:", n_floor)

    log("ragged suffix attention: splits", int(step.desc.n_splits) or "auto")
    step.attention(stream)
    torch.cuda.synchronize()
    got_o = bits_to_f64(host_bits(step.out[LAYERS]))
    sel = []
    for s_i in range(bw.n_seqs):
        sel += [s_i * nq, s_i * nq + nq // 2, s_i * nq + nq - 1]
    sel = np.array(sel)
    errs = []
    for i in range(len(LAYERS)):
        for s_i, sq in enumerate(plan["seqs"]):
            rows = sel[(sel >= s_i * nq) & (sel < (s_i + 1) * nq)]
            base, kvl = sq["seq_base"], sq["kv_len"]
            o, _ = oracle.attention(np.ascontiguousarray(q[i][rows]), np.ascontiguousarray(want_k[i][:, base: base + kvl]),
                                    np.ascontiguousarray(want_v[i][:, base: base + kvl]), q_pos[rows], kvl, bw.scale)
            errs.append((got_o[i][rows], o))
    g = np.concatenate([e[0] for e in errs])
    o = np.concatenate([e[1] for e in errs])
    check_attention_close(g, o)
