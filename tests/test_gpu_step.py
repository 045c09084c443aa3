"""N-block step with selective weight offloading (xema_dit_step_fwd) and
whole-step plans (xema_dit_step_fwd_planned) on the GPU: the output is
bit-identical for every offload plan, staging depth, copy-stream choice,
batch group and chunk size, and to the unserialized, unoffloaded step;
each block matches the fp64 oracle given the GPU's own input to that block
(so a block run with another block's weights, or with half-copied weights,
fails); one block equals the block API."""
import numpy as np
import pytest
import torch

import paper_2607_11136_amd as X
import workloads as W
from oracle import block as O

from gpu_util import DEV, assert_parity, bf16_dev, cfg_of, poison, req_of

pytestmark = pytest.mark.gpu

SHAPE = W.tiny_shape(name="step_d64", cfg_id=70, batch=4, text_len=21, grid=(2, 5, 7), hidden=256,
                     heads=4, head_dim=64, mlp_hidden=512, cond_dim=256, rope_dims=(16, 24, 24))
N = 5


class Stack:
    """Inputs of an N-block step: device and pinned host copies of every
    block's weights."""

    def __init__(self, s, n):
        self.s, self.n = s, n
        self.inputs = W.make_inputs(s)
        self.bits = W.step_weights(s, n)
        self.x, self.cond = bf16_dev(self.inputs.x), bf16_dev(self.inputs.cond)
        self.dev = [{k: bf16_dev(v) for k, v in w.items()} for w in self.bits]
        self.host = []
        for w in self.bits:
            hw = {}
            for k, v in w.items():
                t = torch.empty(v.shape, dtype=torch.bfloat16, pin_memory=True)
                t.copy_(torch.from_numpy(np.ascontiguousarray(v).view(np.int16)).view(torch.bfloat16))
                assert t.data_ptr() % 16 == 0
                hw[k] = t
            self.host.append(hw)
        self.cfg, self.req = cfg_of(s), req_of(s)

    def run(self, n, k, staging=2, chunk=0, copy_stream=None):
        plan = X.xema_offload_plan_k(self.cfg, n, k, staging)
        off = set(plan.offloaded_blocks())
        ws_list = [X.block_weights(self.host[i] if i in off else self.dev[i]) for i in range(n)]
        nbytes = X.xema_step_workspace_bytes(self.cfg, self.req, chunk, plan)
        ws = poison(torch.empty(nbytes, dtype=torch.uint8, device=DEV))
        out = poison(torch.empty((self.s.batch, self.s.seq_len, self.s.hidden), dtype=torch.float32, device=DEV))
        X.xema_dit_step_fwd(self.cfg, self.req, self.x, ws_list, plan, self.cond, chunk, ws, nbytes, out,
                            copy_stream=copy_stream)
        torch.cuda.synchronize()
        return out

    def run_plan(self, plan, copy_stream=None):
        """The step by a whole-step plan (xema_step_plan_fixed / _budget)."""
        n = plan.offload.n_blocks
        off = set(plan.offload.offloaded_blocks())
        ws_list = [X.block_weights(self.host[i] if i in off else self.dev[i]) for i in range(n)]
        ws = poison(torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV))
        out = poison(torch.empty((self.s.batch, self.s.seq_len, self.s.hidden), dtype=torch.float32, device=DEV))
        X.xema_dit_step_fwd_planned(self.cfg, self.req, self.x, ws_list, plan, self.cond, ws, plan.workspace_bytes,
                                    out, copy_stream=copy_stream)
        torch.cuda.synchronize()
        return out


_stack = {}


def _get():
    if "s" not in _stack:
        _stack["s"] = Stack(SHAPE, N)
    return _stack["s"]


def test_step_bit_identical_across_offload_plans():
    st = _get()
    side = torch.cuda.Stream()
    base = st.run(N, 0)
    for k, staging, cs, chunk in ((1, 1, None, 0), (2, 1, side, 0), (2, 2, side, 0), (3, 2, side, 0),
                                  (5, 1, side, 0), (5, 2, None, 0), (5, 3, side, 0), (2, 2, side, 7),
                                  (5, 2, side, 64), (0, 2, None, 100)):
        out = st.run(N, k, staging, chunk, cs)
        assert torch.equal(out, base), (k, staging, cs is not None, chunk)
    # again on the same stream order, reusing the staging slots of the last call
    assert torch.equal(st.run(N, 5, 2, 0, side), base)


def test_step_blocks_match_oracle_given_their_inputs():
    st = _get()
    s = st.s
    kw = dict(heads=s.heads, head_dim=s.head_dim, text_len=s.text_len, grid=s.grid,
              rope_dims=s.rope_dims, rope_theta=s.rope_theta, ln_eps=s.ln_eps, qk_eps=s.qk_eps)
    prev = st.inputs.f64("x")
    cond = st.inputs.f64("cond")
    for n in range(1, N + 1):
        out = st.run(n, n // 2, 2, 0, torch.cuda.Stream()).cpu().numpy().astype(np.float64)
        w = {k: W.bf16_bits_to_f64(v) for k, v in st.bits[n - 1].items()}
        ref = O.block_forward(prev, cond, w, **kw)
        assert_parity(out, ref, f"step block {n - 1} (of {n}, {n // 2} offloaded)")
        prev = out


def test_one_block_step_equals_block_api():
    st = _get()
    out = st.run(1, 1, 1, 0, torch.cuda.Stream())
    plan = X.xema_workspace_layout(st.cfg, st.req, 0)
    ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=DEV)
    ref = torch.empty_like(out)
    X.xema_dit_block_fwd(st.cfg, st.req, st.x, X.block_weights(st.dev[0]), st.cond, 0, ws, ws.numel(), ref)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)


def test_planned_step_bit_identical_to_the_unmitigated_step():
    """Every (K, staging, group, chunk) of the whole-step plan gives the bytes
    of the step with every block resident, the batch whole and no chunks."""
    st = _get()
    side = torch.cuda.Stream()
    base = st.run(N, 0)
    for k, staging, g, chunk in ((0, 2, 4, 0), (0, 2, 2, 0), (0, 2, 1, 0), (2, 2, 2, 64), (5, 1, 1, 7),
                                 (3, 2, 4, 100), (5, 2, 2, 0), (1, 2, 1, 33)):
        plan = X.xema_step_plan_fixed(st.cfg, st.req, N, k, staging, g, chunk)
        print(f"planned step K={k} S={staging} g={g} c={chunk}: workspace {plan.workspace_bytes}", flush=True)
        assert torch.equal(st.run_plan(plan, side), base), (k, staging, g, chunk)


def test_budget_plan_drives_the_planned_step():
    st = _get()
    base = st.run(N, 0)
    free = X.xema_step_plan_fixed(st.cfg, st.req, N, 0, 2, st.s.batch, 0)
    tight = X.xema_step_plan_fixed(st.cfg, st.req, N, N, 2, 1, 0)   # (91 tokens: the only chunk candidate)
    for budget in (free.device_bytes, (free.device_bytes + tight.device_bytes) // 2, tight.device_bytes):
        plan = X.xema_step_plan_budget(st.cfg, st.req, N, 2, budget)
        assert plan.device_bytes <= budget
        print(f"budget {budget}: K={plan.offload.n_offloaded} g={plan.batch_group} c={plan.chunk_tokens}",
              flush=True)
        assert torch.equal(st.run_plan(plan, torch.cuda.Stream()), base), budget


def test_planned_step_blocks_match_oracle_given_their_inputs():
    """Groups of one sequence, chunks of 50 tokens, some blocks offloaded:
    each block against the oracle on the GPU's own input to it."""
    st = _get()
    s = st.s
    kw = dict(heads=s.heads, head_dim=s.head_dim, text_len=s.text_len, grid=s.grid,
              rope_dims=s.rope_dims, rope_theta=s.rope_theta, ln_eps=s.ln_eps, qk_eps=s.qk_eps)
    prev = st.inputs.f64("x")
    cond = st.inputs.f64("cond")
    for n in range(1, 4):
        plan = X.xema_step_plan_fixed(st.cfg, st.req, n, n // 2, 2, 1, 50)
        out = st.run_plan(plan, torch.cuda.Stream()).cpu().numpy().astype(np.float64)
        w = {k: W.bf16_bits_to_f64(v) for k, v in st.bits[n - 1].items()}
        ref = O.block_forward(prev, cond, w, **kw)
        assert_parity(out, ref, f"planned step block {n - 1} (of {n}, g=1, c=50)")
        prev = out


def test_planned_step_refuses_a_foreign_plan():
    st = _get()
    plan = X.xema_step_plan_fixed(st.cfg, st.req, N, 2, 2, 2, 64)
    plan.workspace_bytes -= 256
    ws = torch.empty(1 << 20, dtype=torch.uint8, device=DEV)
    out = torch.empty((st.s.batch, st.s.seq_len, st.s.hidden), dtype=torch.float32, device=DEV)
    with pytest.raises(X.XemaError) as e:
        X.xema_dit_step_fwd_planned(st.cfg, st.req, st.x, [X.block_weights(w) for w in st.dev], plan, st.cond,
                                    ws, ws.numel(), out)
    assert e.value.status == X.XEMA_ERR_INVALID_ARG
