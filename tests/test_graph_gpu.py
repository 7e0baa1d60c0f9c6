"""The hot path captured in a HIP graph (torch.cuda.CUDAGraph on ROCm).

The entry points only enqueue kernels on the caller's stream (no allocation,
no memset, no synchronisation), so a step of PTF-LayerNorm + fused LIS head
can be captured once and replayed.  Each replay runs on new input values
copied into the captured buffers, with eager calls and synchronisations
between replays, and must equal the eager result bit for bit (the eager path
itself is checked against the oracle in test_parity_gpu)."""
import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fq():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2111_13824_amd as fq
    return fq


def say(*a):
    print("CASE", *a, flush=True)


# deit_small_b8 takes the tile kernels of the head, vit_base16_224_b64 the
# unit kernel the benchmark times
@pytest.mark.parametrize("name", ["deit_small_b8", "vit_base16_224_b64"])
def test_step_replayed_from_graph(fq, name):
    import torch
    say("graph", name)
    cfg = W.BY_NAME[name]
    inp = W.config_inputs(cfg)
    ln, at = inp["ln"], inp["attn"]
    d = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to("cuda:0")
    x0, lg0, v0 = d(ln["x_q"]), d(at["logits"]), d(at["v"])
    alpha, gamma, beta = d(ln["alpha"]), d(ln["gamma"]), d(ln["beta"])
    x, lg, v = x0.clone(), lg0.clone(), v0.clone()
    y = torch.empty_like(x)
    out = torch.empty((cfg.G, cfg.Lq, cfg.d), dtype=torch.int32, device="cuda:0")

    def step(y_q, o):
        fq.ptf_layernorm_int8(x, ln["zp_in"], alpha, ln["K"], gamma, beta, ln["s_out"],
                              ln["zp_out"], ln["bits"], y_q=y_q)
        fq.lis_attention_head(lg, v, at["s_logit"], at["bits"], at["exp_n"], zp_v=at["zp_v"],
                              out=o)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(y, out)                      # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(y, out)
    torch.cuda.synchronize()

    y_e = torch.empty_like(y)
    o_e = torch.empty_like(out)
    for rep in range(4):
        # new values in the captured buffers: rows and units rolled, V negated
        x.copy_(torch.roll(x0, shifts=97 * rep, dims=0))
        lg.copy_(torch.roll(lg0, shifts=5 * rep, dims=0))
        v.copy_(v0 if rep % 2 == 0 else torch.clamp(-v0.to(torch.int16), -128, 127).to(torch.int8))
        y.fill_(0)
        out.fill_(-1)
        g.replay()
        torch.cuda.synchronize()
        step(y_e, o_e)                    # eager on the same inputs
        torch.cuda.synchronize()
        assert torch.equal(y, y_e), f"LayerNorm replay {rep}"
        assert torch.equal(out, o_e), f"head replay {rep}"
