"""The allocation-free attention entry point (kvlink_attend_new_tokens_noalloc)
against the entry point that takes a workspace: the same kernels and schedule
over the library's own scratch, so the outputs and LSE must be equal bit for
bit.  Three calls in a row on one stream, each smaller than the one before
(the 10-document Llama-8B layer with split partials, a ragged bf16 batch on
the decode kernel, the tiny fp32 workload on the vector kernel): the scratch
keeps the previous call's bytes, and no call may read them."""
import numpy as np
import pytest

import workloads
from harness import ContiguousRun

pytestmark = pytest.mark.gpu


def _noalloc(run, l, out, lse):
    import paper_2502_16002_amd as kv
    b = run.batch
    kv.kvlink_attend_new_tokens_noalloc(
        b.dtype, b.n_q_heads, b.n_kv_heads, b.head_dim, b.rope_theta, b.softmax_scale, b.n_seqs,
        b.n_new, b.max_new, b.max_cached, b.d_seq_new_ptr, b.d_seq_cached, b.d_new_pos,
        b.d_new_visible, run.q[l], run.kn[l], run.vn[l], run.k_view, run.v_view, l, out, lse,
        b.plan)


def test_noalloc_matches_workspace_entry_point_on_successive_smaller_calls():
    import torch
    import paper_2502_16002_amd as kv
    runs = [ContiguousRun(workloads.llama8b_10doc(n_layers=1), layers=[0]),
            ContiguousRun(workloads.custom([130, 5, 260], [1, 0, 1], 2, n_q_heads=8, n_kv_heads=2,
                                           head_dim=128, dtype="bf16", rope_theta=5e5, seed=23),
                          layers=[0]),
            ContiguousRun(workloads.tiny_f32(), layers=[0])]
    need = [kv.kvlink_attend_workspace_bytes(r.batch.dtype, r.batch.n_q_heads,
                                             r.batch.n_kv_heads, r.batch.head_dim, r.batch.n_new,
                                             r.batch.plan) for r in runs]
    print("scratch bytes per call", need, flush=True)
    assert need[0] > need[1] > need[2] and need[0] <= kv.KVLINK_NOALLOC_SCRATCH_BYTES
    assert runs[0].batch.plan.n_split_units > 0          # the first call writes split partials
    for r in runs:
        r.run()                                          # workspace entry point: out[0], lse[0]
    got = []
    for r in runs:                                       # back to back, one stream, no sync
        out, lse = r.batch.new_out(), r.batch.new_lse()
        _noalloc(r, 0, out, lse)
        got.append((out, lse))
    torch.cuda.synchronize()
    for r, (out, lse) in zip(runs, got):
        assert torch.equal(out.view(torch.int16) if out.dtype == torch.bfloat16 else out,
                           r.out[0].view(torch.int16) if out.dtype == torch.bfloat16 else r.out[0]), r.w.name
        assert torch.equal(lse, r.lse[0]), r.w.name
        print(r.w.name, "noalloc == workspace entry point", flush=True)
    # the same again in the opposite order of sizes is just as exact
    for r in reversed(runs):
        out, lse = r.batch.new_out(), r.batch.new_lse()
        _noalloc(r, 0, out, lse)
        torch.cuda.synchronize()
        assert torch.equal(lse, r.lse[0]), r.w.name
