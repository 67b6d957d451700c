"""The whole step against the oracle: route on X, compress, reconstruct, experts on X_hat."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2508_06024_amd import workload as W
from paper_2508_06024_amd.layer import Ec2moeLayer
from tests.gpu_common import assert_close, check_routing, down, say, tol, up, up_f32

pytestmark = pytest.mark.gpu


def build(inp, top_groups=0, group_sizes=None):
    cfg = inp.cfg
    dt = cfg.dtype
    return Ec2moeLayer(up(inp.x, dt), inp.mask, up(inp.w_global, dt), up_f32(inp.b_global), up(inp.w_local, dt),
                       up_f32(inp.b_local), up(inp.w_gate_up, dt), up(inp.w_down, dt), up(inp.u, dt),
                       up(inp.v, dt), n_groups=cfg.n_groups, top_k=cfg.top_k, activation=cfg.activation,
                       codec_slices=cfg.codec_slices, top_groups=top_groups, group_sizes=group_sizes)


def oracle_sampled(inp, toks, top_groups=0, group_sizes=None):
    """Oracle layer outputs of the sampled tokens: the gate and the experts act per token;
    the codec's Z couples all tokens of a slice and is computed in full, slice by slice."""
    cfg = inp.cfg
    f = inp.f64
    x, u, v = f("x"), f("u"), f("v")
    idx, w, g = O.group_gate(x[toks], f("w_global"), inp.b_global, f("w_local"), inp.b_local, inp.mask,
                             cfg.n_groups, cfg.top_k, group_sizes=group_sizes, top_groups=top_groups)
    h = cfg.codec_h
    z = np.stack([O.lowrank_encode(x[s * h:(s + 1) * h], u, v) for s in range(cfg.codec_slices)])
    if len(toks) == cfg.n_tokens:
        xh = np.concatenate([O.lowrank_decode(z[s], u, v) for s in range(cfg.codec_slices)])
    else:
        xh = np.stack([O.lowrank_decode(z[t // h], u[[t % h]], v)[0] for t in toks])
    y = np.zeros((len(toks), cfg.d_model))
    expert = O.EXPERTS[cfg.activation]
    for e in np.unique(idx):
        gu = W.to_f64(inp.w_gate_up[e], cfg.dtype)
        dn = W.to_f64(inp.w_down[e], cfg.dtype)
        rows, slots = np.nonzero(idx == e)
        y[rows] += w[rows, slots, None] * expert(xh[rows], gu, dn)
    return idx, w, g, z, xh, y


@pytest.mark.parametrize("name,call", [("tiny", None), ("small", None), ("mixtral", None), ("finegrained", None),
                                       ("decode", 4), ("decode", 777), ("switch8", None), ("switch16", None),
                                       ("switch32", None), ("switch64", None)])
def test_layer_step_matches_oracle(name, call):
    """Every token of the step: routing (certified near-ties aside), Z, X_hat and y."""
    cfg = W.CONFIGS[name]
    say(f"layer {name} call {call}")
    torch.cuda.empty_cache()
    inp = W.gen_layer(cfg, call_seed=call)
    lay = build(inp)
    lay.step()
    torch.cuda.synchronize()
    toks = np.arange(cfg.n_tokens)
    idx, w, g, z, xh, y = oracle_sampled(inp, toks)
    gidx, gw = down(lay.topk_idx)[toks], down(lay.topk_w)[toks]
    n_cert = check_routing(gidx, gw, idx, w, g, W.mask_members(inp.mask, cfg.n_experts), cfg.top_k)
    assert_close(down(lay.z).reshape(z.shape), z, 1e-5, "Z")
    assert_close(down(lay.x_hat)[toks], xh, tol(cfg.dtype), "X_hat")
    same = ~(gidx != idx).any(axis=1)
    e = assert_close(down(lay.y)[toks][same], y[same], tol(cfg.dtype), "y")
    say(f"  y rel err {e:.2e}; certified near-ties {n_cert}")
    # same inputs, same bits
    y1 = lay.y.clone()
    lay.step()
    assert torch.equal(lay.y, y1)


def test_layer_step_with_unequal_groups_and_top_groups():
    """The whole step with groups of unequal sizes (K does not divide M) and group-focused
    evaluation (the top 2 groups per token): the calls after the gate take any K <= M."""
    from tests.test_gpu_gate import _group_cut_near_ties
    cfg = W.LayerConfig("unequal", W.BF16, 300, 1024, 24, 5, 256, 3, 32, 32, seed=17, mask="random", n_keep=18,
                        x_dist="rms", gate_std=0.05)
    sizes, G = (2, 7, 3, 8, 4), 2
    say(f"layer unequal groups {sizes} top_groups {G}")
    inp = W.gen_layer(cfg)
    lay = build(inp, top_groups=G, group_sizes=sizes)
    lay.step()
    torch.cuda.synchronize()
    toks = np.arange(cfg.n_tokens)
    idx, w, g, z, xh, y = oracle_sampled(inp, toks, top_groups=G, group_sizes=sizes)
    members = W.mask_members(inp.mask, cfg.n_experts)
    amb = _group_cut_near_ties(inp.x, inp.w_global, inp.b_global, members, cfg.n_experts, cfg.n_groups, cfg.top_k,
                               sizes, G)
    assert amb.size <= 0.05 * cfg.n_tokens
    ok = np.setdiff1d(toks, amb)
    gidx, gw = down(lay.topk_idx), down(lay.topk_w)
    check_routing(gidx[ok], gw[ok], idx[ok], w[ok], g[ok], members, cfg.top_k)
    assert_close(down(lay.z).reshape(z.shape), z, 1e-5, "Z")
    same = ~(gidx != idx).any(axis=1)
    same[amb] = False
    e = assert_close(down(lay.y)[same], y[same], tol(cfg.dtype), "y")
    say(f"  y rel err {e:.2e}; tokens with near-tied groups at the cut {amb.size}")


@pytest.mark.parametrize("name", ["small", "decode"])
def test_overlapped_routing_matches_one_stream_order(name):
    """The routing on its own stream (the default) gives the one-stream order's bits, step
    after step, with the input and the candidate mask changing between steps."""
    cfg = W.CONFIGS[name]
    say(f"overlapped routing {name}")
    inp = W.gen_layer(cfg, call_seed=5 if cfg.mask == "per_call" else None)
    dt = cfg.dtype
    per_call = cfg.mask == "per_call"
    calls = [W.gen_call(cfg, call_seed=10 + j) if per_call else W.gen_call(cfg.scaled(seed=cfg.seed + j))
             for j in (1, 2, 3)]
    xs = [up(c[0], dt) for c in calls]
    masks = [c[1] for c in calls]
    kw = dict(n_groups=cfg.n_groups, top_k=cfg.top_k, activation=cfg.activation, codec_slices=cfg.codec_slices)
    args = (up(inp.x, dt), inp.mask, up(inp.w_global, dt), up_f32(inp.b_global), up(inp.w_local, dt),
            up_f32(inp.b_local), up(inp.w_gate_up, dt), up(inp.w_down, dt), up(inp.u, dt), up(inp.v, dt))
    seq = Ec2moeLayer(*args, overlap=False, **kw)
    ovl = Ec2moeLayer(*args, overlap=True, **kw)
    for step in range(6):
        x, m = xs[step % 3], masks[step % 3]
        for lay in (seq, ovl):
            lay.set_input(x, m)
            lay.step()
        torch.cuda.synchronize()
        for a, b in ((seq.y, ovl.y), (seq.topk_idx, ovl.topk_idx), (seq.topk_w, ovl.topk_w), (seq.z, ovl.z)):
            assert torch.equal(a, b), f"step {step}"
