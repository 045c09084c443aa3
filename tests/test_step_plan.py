"""The N-block step's static layout and whole-step plan (CPU only): the
library's planner (csrc/step_plan.cpp, through the C ABI) against the
oracle (oracle/step_plan.py), the layout's validity, the latency model's
closed forms and the plan's "only as much as needed" behaviour."""
import itertools
import math

import pytest

import oracle.layout as LY
import oracle.offload as OF
import oracle.step_plan as SP
import paper_2607_11136_amd as X
import workloads as W

# small shapes: several batch groups, a ragged chunk, both head widths
SHAPES = {
    "b4_d64": W.tiny_shape(name="sp_b4", cfg_id=80, batch=4, text_len=20, grid=(2, 10, 15), hidden=256, heads=4,
                           head_dim=64, mlp_hidden=1024, cond_dim=256, rope_dims=(16, 24, 24)),
    "b2_d128": W.tiny_shape(name="sp_b2", cfg_id=81, batch=2, text_len=7, grid=(1, 12, 20), hidden=512, heads=4,
                            head_dim=128, mlp_hidden=1536, cond_dim=512, rope_dims=(0, 64, 64)),
    "b1_tiny": W.TINY,
}
COSTS = (56.0, 1000.0)


def _cfg(s):
    return X.block_cfg(s.hidden, s.heads, s.head_dim, s.mlp_hidden, s.cond_dim, s.rope_dims, s.rope_theta,
                       s.ln_eps, s.qk_eps, s.modulation_streams, s.weights_f16)


def _req(s):
    return X.request(s.batch, s.text_len, *s.grid)


def _slot_bytes(s):
    return OF.slot_bytes(OF.block_weight_sizes(s.hidden, s.mlp_hidden, s.cond_dim, s.head_dim,
                                               s.modulation_streams))


def _groups(b):
    return [g for g in range(b, 0, -1) if b % g == 0]


@pytest.mark.parametrize("name", sorted(SHAPES))
def test_step_layout_matches_oracle(name):
    s = SHAPES[name]
    for n, k, g, c in itertools.product((1, 2, 3, 5), (0, 1, 3), _groups(s.batch), (0, 64, 257)):
        if k > n:
            continue
        p = X.xema_step_plan_fixed(_cfg(s), _req(s), n, k, 2, g, c, X.step_costs(*COSTS))
        want = SP.plan_fixed(s, n, k, 2, g, c, *COSTS)
        assert p.workspace_bytes == want["workspace_bytes"], (name, n, k, g, c)
        assert p.device_bytes == want["device_bytes"]
        assert math.isclose(p.est_ms, want["est_ms"], rel_tol=1e-12), (p.est_ms, want["est_ms"])
        assert p.batch_group == g and p.chunk_tokens == want["chunk"]
        assert p.offload.offloaded_blocks() == want["offloaded"]


def _check_valid(ts, offs):
    for a, b in itertools.combinations(range(len(ts)), 2):
        if LY.overlaps(ts[a], ts[b]) and ts[a].size and ts[b].size:
            ra = (offs[a], offs[a] + LY.round_up(ts[a].size, LY.ALIGN))
            rb = (offs[b], offs[b] + LY.round_up(ts[b].size, LY.ALIGN))
            assert ra[1] <= rb[0] or rb[1] <= ra[0], (ts[a], ts[b], ra, rb)


@pytest.mark.parametrize("name", sorted(SHAPES))
def test_step_layout_is_valid_and_not_above_the_concatenation(name):
    """No two tensors alive together share bytes; the peak reaches at least
    the max-live bound and at most the concatenation [block arena | one
    residual buffer | staging slots] that a layout without Algorithm 1 over
    the step would take."""
    s = SHAPES[name]
    slot = _slot_bytes(s)
    for n, g, c, st in itertools.product((1, 2, 4, 7), _groups(s.batch), (0, 100), (0, 2)):
        ts, what = SP.step_tensors(s, n, g, c, st, slot)
        offs, peak = LY.static_layout(ts)
        _check_valid(ts, offs)
        assert peak >= LY.max_live_bytes(ts)
        arena = LY.workspace_bytes(s.with_(batch=g), c)
        resid = 4 * s.batch * s.seq_len * s.hidden if n > 1 else 0
        assert peak <= arena + LY.round_up(resid, LY.ALIGN) + st * slot, (name, n, g, c, st)
        # the buffers of block i's output alternate with the caller's out
        assert sorted(w[1] for w in what.values() if w[0] == "resid") == \
            [i for i in range(n - 1) if (n - 1 - i) % 2 == 1]


def test_unserialized_step_workspace_is_the_plan_layout():
    s = SHAPES["b4_d64"]
    for n, k, c in ((1, 0, 0), (4, 2, 64), (6, 6, 0)):
        op = X.xema_offload_plan_k(_cfg(s), n, k, 2)
        got = X.xema_step_workspace_bytes(_cfg(s), _req(s), c, op)
        assert got == X.xema_step_plan_fixed(_cfg(s), _req(s), n, k, 2, s.batch, c).workspace_bytes


def test_latency_model_closed_forms():
    t_blk, t_x = 3.0, 5.0
    # no offloading: the blocks back to back
    assert SP.step_ms(6, [], 2, t_blk, t_x) == 6 * t_blk
    # every block offloaded through one staging slot: each copy waits for the
    # block before it, nothing overlaps
    assert SP.step_ms(4, [0, 1, 2, 3], 1, t_blk, t_x) == 4 * (t_x + t_blk)
    # two slots and copies shorter than a block: one copy exposed, then pipelined
    assert SP.step_ms(5, [0, 1, 2, 3, 4], 2, 4.0, 2.0) == 2.0 + 5 * 4.0
    # one offloaded block at the end of the stack, its copy hidden behind the others
    assert SP.step_ms(5, [4], 2, t_blk, t_x) == 5 * t_blk
    # the library's simulation agrees on the same plans
    s = SHAPES["b1_tiny"]
    for n, k, st in ((6, 0, 2), (4, 4, 1), (5, 5, 2), (5, 1, 2), (7, 3, 2)):
        p = X.xema_step_plan_fixed(_cfg(s), _req(s), n, k, st, 1, 0, X.step_costs(*COSTS))
        t_b = SP.block_ms(s, 1, 0, COSTS[1])
        t_c = _slot_bytes(s) / (COSTS[0] * 1e9) * 1e3
        assert math.isclose(p.est_ms, SP.step_ms(n, p.offload.offloaded_blocks(), p.offload.n_staging, t_b, t_c),
                            rel_tol=1e-12)


def test_block_model_never_favours_a_smaller_launch():
    """Rounds of split launches are never fewer than those of the whole:
    chunking and serialization cost time in the model, never save it."""
    for s in (SHAPES["b4_d64"], W.VIDEO, W.IMAGE_B4):
        full = SP.block_ms(s, s.batch, 0, 1000.0)
        assert full >= s.flops() / 1e15 * 1e3 * (1 - 1e-9)    # at least the FLOPs at the rate
        for g in _groups(s.batch):
            for c in (0, 4096, 1000, 256):
                assert SP.block_ms(s, g, c, 1000.0) >= full * (1 - 1e-12), (s.name, g, c)


@pytest.mark.parametrize("name", ["b4_d64", "b2_d128"])
def test_budget_plan_matches_oracle(name):
    s = SHAPES[name]
    n = 4
    free = SP.plan_fixed(s, n, 0, 2, s.batch, 0, *COSTS)["device_bytes"]
    least = min(SP.plan_fixed(s, n, n, 2, 1, c, *COSTS)["device_bytes"] for c in LY.chunk_candidates(s.seq_len))
    for budget in sorted({free, free - 1, (free + least) // 2, least + 4096, least}):
        want = SP.plan_budget(s, n, 2, budget, *COSTS)
        got = X.xema_step_plan_budget(_cfg(s), _req(s), n, 2, budget, X.step_costs(*COSTS))
        assert want is not None
        assert (got.offload.n_offloaded, got.batch_group, got.chunk_tokens) == \
            (want["k"], want["group"], want["chunk"]), (budget, want)
        assert got.device_bytes == want["device_bytes"] <= budget
        assert math.isclose(got.est_ms, want["est_ms"], rel_tol=1e-12)
    with pytest.raises(X.XemaError) as e:
        X.xema_step_plan_budget(_cfg(s), _req(s), n, 2, least - 1, X.step_costs(*COSTS))
    assert e.value.status == X.XEMA_ERR_BUDGET_TOO_SMALL and e.value.plan.device_bytes == least


def test_ample_budget_takes_no_mitigation_and_tight_budgets_take_some():
    s = SHAPES["b4_d64"]
    n = 6
    free = X.xema_step_plan_fixed(_cfg(s), _req(s), n, 0, 2, s.batch, 0)
    p = X.xema_step_plan_budget(_cfg(s), _req(s), n, 2, free.device_bytes)
    assert (p.offload.n_offloaded, p.batch_group, p.chunk_tokens) == (0, s.batch, s.seq_len)
    assert p.est_ms == free.est_ms
    q = X.xema_step_plan_budget(_cfg(s), _req(s), n, 2, free.device_bytes - 1)
    assert (q.offload.n_offloaded, q.batch_group, q.chunk_tokens) != (0, s.batch, s.seq_len)
    assert q.device_bytes < free.device_bytes and q.est_ms >= free.est_ms


def test_video_step_plans_under_one_budget():
    """Twenty video blocks (17,776 tokens): an ample budget runs everything
    resident and unchunked; budgets that leave room for few blocks' weights
    trade offloading against chunking by the model, every plan within its
    budget and never modelled faster than the unmitigated step."""
    s = W.VIDEO
    n = 20
    cfg, req = _cfg(s), _req(s)
    free = X.xema_step_plan_fixed(cfg, req, n, 0, 2, 1, 0)
    prev = None
    for frac in (1.0, 0.8, 0.6, 0.4, 0.25):
        budget = int(free.device_bytes * frac)
        p = X.xema_step_plan_budget(cfg, req, n, 2, budget)
        assert p.device_bytes <= budget and p.est_ms >= free.est_ms * (1 - 1e-12)
        if prev is not None:
            assert p.est_ms >= prev.est_ms * (1 - 1e-12)   # less memory never models faster
        prev = p


# -- the layout against the step's operations in their real order -------------------------------

SLOT = {n: i for i, n in enumerate(LY.SLOT_NAMES)}


def _replay(s, n, g, c):
    """Live instances (buffer, first write, last read) of every buffer the
    step's workspace holds, in the order the step runs its operations:
    blocks, then groups of g sequences, then phase A per chunk (LN1; QKV
    writing Q, K, V^T) and phase B per chunk (attention; out-projection
    reading the block's input; LN2; MLP up; MLP down writing the block's
    output).  A buffer rewritten per group or per chunk starts a new
    instance each time; the block's input is one instance from its first
    write in the previous block to its last read."""
    B, L = s.batch, s.seq_len
    c = L if c <= 0 or c >= L else c
    chunks = list(range(0, L, c))
    t = 0
    spans = []
    resid_first, resid_last = {}, {}

    def out_key(i):
        return ("resid", i) if (n - 1 - i) % 2 == 1 else None

    for i in range(n):
        x_in = out_key(i - 1) if i > 0 else None
        for _ in range(B // g):
            t += 1
            start = t                                   # AdaLN map, RoPE table, status clear
            qkv_start = None
            for _ in chunks:
                t += 1
                ln1 = t                                 # LN1 reads the input, writes ln1
                if x_in:
                    resid_last[x_in] = t
                t += 1                                  # QKV reads ln1, writes Q, K, V^T
                spans.append((("slot", i, SLOT["ln1"]), ln1, t))
                qkv_start = qkv_start or t
            spans.append((("slot", i, SLOT["rope"]), start, t))
            t += 1
            copies = t                                  # the fp16 weight copies
            for _ in chunks:
                t += 1
                attn = t                                # attention reads Q, K, V^T
                qkv_end = t
                t += 1                                  # out-projection reads attn and the input
                spans.append((("slot", i, SLOT["attn"]), attn, t))
                x1 = t
                if x_in:
                    resid_last[x_in] = t
                t += 1
                ln2 = t
                t += 1
                spans.append((("slot", i, SLOT["ln2"]), ln2, t))
                hid = t
                t += 1                                  # MLP down reads hid and x1, writes the output
                spans.append((("slot", i, SLOT["hid"]), hid, t))
                spans.append((("slot", i, SLOT["x1"]), x1, t))
                if out_key(i):
                    resid_first.setdefault(out_key(i), t)
            for name in ("q", "k", "vt"):
                spans.append((("slot", i, SLOT[name]), qkv_start, qkv_end))
            for name in ("wo16", "wup16", "wdown16"):
                spans.append((("slot", i, SLOT[name]), copies, t))
            for name in ("mod", "status"):
                spans.append((("slot", i, SLOT[name]), start, t))
    for key, first in resid_first.items():
        spans.append((key, first, resid_last[key]))
    return spans


@pytest.mark.parametrize("name", sorted(SHAPES))
def test_step_layout_respects_the_real_order_of_operations(name):
    s = SHAPES[name]
    slot = _slot_bytes(s)
    for n, g, c in itertools.product((1, 2, 3, 5), _groups(s.batch), (0, 7, 100)):
        ts, what = SP.step_tensors(s, n, g, c, 2, slot)
        offs, _ = LY.static_layout(ts)
        where = {}
        for t, o in zip(ts, offs):
            kind = what[t.sid]
            key = ("slot", kind[1], kind[2]) if kind[0] == "slot" else (("resid", kind[1]) if kind[0] == "resid"
                                                                           else None)
            if key:
                where[key] = (o, o + LY.round_up(t.size, LY.ALIGN))
        spans = [sp for sp in _replay(s, n, g, c) if sp[0] in where]
        for (ka, a0, a1), (kb, b0, b1) in itertools.combinations(spans, 2):
            if ka == kb:
                continue
            ra, rb = where[ka], where[kb]
            if ra[0] < rb[1] and rb[0] < ra[1]:        # they share bytes: never live together
                assert a1 < b0 or b1 < a0, (name, n, g, c, ka, (a0, a1), kb, (b0, b1))
