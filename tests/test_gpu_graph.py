"""HIP-graph capture of the hot path (stream capture through torch.cuda.CUDAGraph): the single-layer step
(window attention with score partials, scores, prune + compaction) on the seq-4096 workload, and a 4-layer
encoder stack.  Each graph is replayed several times, with eager work of the program (poisoning every output
buffer, an unrelated window attention, synchronisations) between the replays, and every replay must reproduce
the eager results bit for bit (the kernels are deterministic)."""
import numpy as np
import pytest
import torch

import sc_inputs as si
from gpu_helpers import DEV, dev_i32, log, make_desc, stored_threshold, to_dev_storage

import paper_2310_07109_amd as sc

pytestmark = pytest.mark.gpu


def _capture(step):
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    return g


def _snapshot(bufs):
    return {k: (v.view(torch.int16) if v.dtype == torch.bfloat16 else v).cpu().numpy().copy() for k, v in bufs.items()}


def _poison(bufs):
    for v in bufs.values():
        if v.dtype in (torch.float32, torch.bfloat16):
            v.fill_(float("nan"))
        else:
            v.fill_(-7)


def _other_attention():
    """Unrelated eager work between replays."""
    inp = si.make_attention_inputs(si.CONFIGS[2], seed=31, B=2, n=512)
    d = make_desc(inp)
    q, k, v = (to_dev_storage(inp[x], "bf16") for x in ("q", "k", "v"))
    sc.sc_window_attention(d, q, k, v)


def test_single_layer_step_graph_replays():
    inp = si.make_attention_inputs(si.CONFIGS[4])
    d = make_desc(inp)
    B, n, H, G = d.B, d.n, d.H, d.G
    theta = stored_threshold(4)
    q, k, v = (to_dev_storage(inp[x], "bf16") for x in ("q", "k", "v"))
    bufs = dict(out=torch.empty_like(q), lse=torch.empty((B, H, n), dtype=torch.float32, device=DEV),
                sp=torch.empty(sc.sc_score_partials_size(d) // 4, dtype=torch.float32, device=DEV),
                scores=torch.empty((B, n), dtype=torch.float32, device=DEV),
                keep=torch.empty((B, n), dtype=torch.int32, device=DEV),
                nl=torch.empty((B,), dtype=torch.int32, device=DEV),
                ngp=torch.empty((B, G), dtype=torch.int32, device=DEV),
                orig=torch.empty((B, n), dtype=torch.int32, device=DEV), oc=torch.empty_like(q))
    ws = torch.empty(sc.sc_window_attention_workspace_size(d), dtype=torch.uint8, device=DEV)
    wsp = torch.empty(sc.sc_ltp_prune_compact_workspace_size(d), dtype=torch.uint8, device=DEV)

    def step():
        sc.sc_window_attention(d, q, k, v, out=bufs["out"], lse=bufs["lse"], score_partials=bufs["sp"], workspace=ws)
        sc.sc_ltp_score(d, bufs["sp"], scores=bufs["scores"])
        sc.sc_ltp_prune_compact(d, bufs["scores"], theta, True, [bufs["out"]], dsts=[bufs["oc"]],
                                outs=dict(keep_idx=bufs["keep"], new_len=bufs["nl"], new_global_pos=bufs["ngp"],
                                          orig_idx_out=bufs["orig"]), workspace=wsp)

    _poison(bufs)
    step()
    torch.cuda.synchronize()
    ref = _snapshot(bufs)
    # compacted rows beyond new_len are unspecified: compare only the written ones
    nl = ref["nl"]
    for b in range(B):
        ref["oc"][b, nl[b]:] = 0
    g = _capture(step)
    for r in range(3):
        _poison(bufs)
        _other_attention()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = _snapshot(bufs)
        for b in range(B):
            got["oc"][b, nl[b]:] = 0
        for key in ref:
            assert np.array_equal(got[key], ref[key], equal_nan=True), f"replay {r}: {key} differs from eager"
        log(f"single-layer step replay {r}: bit-identical to the eager step")


def test_encoder_stack_graph_replays():
    cfg = si.StackConfig("graph stack", 41, 3, 600, 4, 64, 4, 128, (200, 600), 1, 0.05, 0.012)
    inp = si.make_stack_inputs(cfg)
    d = sc.Desc(cfg.B, cfg.n, cfg.H, cfg.window, dev_i32(inp["valid_len"]), dev_i32(inp["global_pos"]), cfg.alpha,
                sc.SC_BF16)
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(DEV).view(torch.bfloat16)  # noqa
    x = bf(inp["x"])
    wq, wo = [bf(w) for w in inp["wqkv"]], [bf(w) for w in inp["wo"]]
    thetas = [0.0, 0.004, 0.008, 0.012]
    x_out = torch.empty_like(x)
    ws = torch.empty(sc.sc_encoder_attn_stack_workspace_size(d, len(thetas)), dtype=torch.uint8, device=DEV)
    res = {}

    def step():
        res["r"] = sc.sc_encoder_attn_stack(d, x, wq, wo, thetas, x_out=x_out, workspace=ws)

    step()
    torch.cuda.synchronize()
    y, fl, orig, kpl = res["r"]
    fl_ref = fl.cpu().numpy().copy()
    ref = dict(fl=fl_ref, orig=orig.cpu().numpy().copy(), kpl=kpl.cpu().numpy().copy(),
               y=np.concatenate([y[b, :fl_ref[b]].view(torch.int16).cpu().numpy().ravel() for b in range(cfg.B)]))
    g = _capture(step)
    y, fl, orig, kpl = res["r"]  # the graph's own output tensors
    for r in range(3):
        for t in (fl, orig, kpl):
            t.fill_(-7)
        x_out.fill_(float("nan"))
        _other_attention()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got_fl = fl.cpu().numpy()
        assert np.array_equal(got_fl, ref["fl"]), f"replay {r}: final lengths differ"
        assert np.array_equal(orig.cpu().numpy(), ref["orig"]) and np.array_equal(kpl.cpu().numpy(), ref["kpl"])
        got_y = np.concatenate([x_out[b, :got_fl[b]].view(torch.int16).cpu().numpy().ravel() for b in range(cfg.B)])
        assert np.array_equal(got_y, ref["y"]), f"replay {r}: hidden states differ"
        log(f"stack replay {r}: bit-identical to the eager call (kept per layer {ref['kpl'].sum(axis=1).tolist()})")
