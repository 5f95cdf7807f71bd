"""Concurrent calls on two streams: the batch's sequences as two halves, each half's window attention, scores and
prune + compaction on a stream of its own (each with its own workspaces), give bit-identical results to one call
on the whole batch."""
import numpy as np
import pytest
import torch

import sc_inputs as si
from gpu_helpers import dev_i32, log, to_dev_storage

pytestmark = pytest.mark.gpu

import paper_2310_07109_amd as sc  # noqa: E402


def _run(inp, rows, theta, stream):
    sel = np.array(rows)
    n, H = inp["n"], inp["H"]
    d = sc.Desc(len(rows), n, H, inp["window"], dev_i32(inp["valid_len"][sel]), dev_i32(inp["global_pos"][sel]),
                inp["alpha"], sc.SC_BF16)
    q, k, v = (to_dev_storage(np.ascontiguousarray(inp[x][sel]), "bf16") for x in ("q", "k", "v"))
    with torch.cuda.stream(stream):
        out, lse, sp, _ = sc.sc_window_attention(d, q, k, v, lse=True, score_partials=True, stream=stream)
        scores = sc.sc_ltp_score(d, sp, stream=stream)
        oc = torch.empty_like(out)
        keep_idx, new_len, new_gp, _, _ = sc.sc_ltp_prune_compact(d, scores, theta, True, [out], dsts=[oc],
                                                                  stream=stream)
    return dict(out=out, lse=lse, scores=scores, oc=oc, keep_idx=keep_idx, new_len=new_len, new_gp=new_gp)


def test_two_streams_match_one_call():
    cfg = si.CONFIGS[4]
    inp = si.make_attention_inputs(cfg, B=4, n=2048, len_range=(1024, 2048))
    theta = 3.7e-4
    main = torch.cuda.current_stream()
    whole = _run(inp, list(range(4)), theta, main)
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    halves = [(list(range(0, 4, 2)), s1), (list(range(1, 4, 2)), s2)]
    for _ in range(3):  # repeated, so that the two halves' launches overlap on the device
        res = [_run(inp, rows, theta, st) for rows, st in halves]
        torch.cuda.synchronize()
        for (rows, _), r in zip(halves, res):
            for j, b in enumerate(rows):
                L = int(inp["valid_len"][b])
                nl = int(whole["new_len"][b])
                assert int(r["new_len"][j]) == nl
                assert torch.equal(r["out"][j, :L].view(torch.int16), whole["out"][b, :L].view(torch.int16))
                assert torch.equal(r["lse"][j, :, :L], whole["lse"][b, :, :L])
                assert torch.equal(r["scores"][j], whole["scores"][b])
                assert torch.equal(r["keep_idx"][j, :nl], whole["keep_idx"][b, :nl])
                assert torch.equal(r["oc"][j, :nl].view(torch.int16), whole["oc"][b, :nl].view(torch.int16))
                assert torch.equal(r["new_gp"][j], whole["new_gp"][b])
    log("two streams: bit-identical to one call over the whole batch")
