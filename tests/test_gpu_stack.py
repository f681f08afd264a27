"""Whole-step parity of the layer stack, in the launch configuration the
benchmark times.

* 64^3 fp32 stack (batch 1): the whole forward chain against the oracle's
  fp64 chain from the same input and weights (gated), and every backward op
  teacher-forced from the tensors the GPU produced (gated).
* 128^3 stacks at full size (fp32 batch 1, bf16 batch 8): sampled outputs of
  every op, each evaluated one by one by the oracle's single-element
  evaluators from the GPU's own inputs to that op.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_1808_04728_amd import binding as B
from paper_1808_04728_amd import inputs
from paper_1808_04728_amd.stack import ConvStack
from tests._util import TOL, maxabs_err, to_np

pytestmark = pytest.mark.gpu


def build(name, fused=True):
    wl = inputs.WORKLOADS[name]
    st = ConvStack(wl["layers"], wl["size"], wl["batch"], wl["dtype"], inputs.ALPHA, "cuda", fused=fused)
    ws, bs = inputs.make_weights(name)
    st.set_params(ws, bs)
    st.set_input(inputs.make_input(name))
    dout = torch.as_tensor(inputs.normal((wl["batch"],) + st.out_dhw + (wl["layers"][-1]["cout"],),
                                         30000 + wl["cfg"]), device="cuda").to(st.tdt)
    return wl, st, dout


def mask_bits(l):
    od = l["out_dhw"]
    n = l["nvox"] * l["spec"]["cout"]
    bits = np.unpackbits(l["mask"].cpu().numpy().view(np.uint8), bitorder="little")[:n]
    return bits.astype(bool).reshape((-1,) + tuple(od) + (l["spec"]["cout"],))


def fused_dz(l, g, alpha):
    """dz of a fused pooled layer, rebuilt from its pooled gradient and mask."""
    dy = oracle.avgpool3d_bwd(to_np(g), l["out_dhw"])
    return dy * np.where(mask_bits(l), 1.0, alpha)


@pytest.mark.parametrize("name", ["stack_64c_b1_f32", "paper_c1c3_64_b1_f32"])
@pytest.mark.parametrize("fused", [True, False])
def test_stack_64_f32_chain(fused, name):
    """The SAME-padded stack and the paper's VALID first three layers."""
    wl, st, dout = build(name, fused)
    st.forward()
    st.backward(dout)
    torch.cuda.synchronize()
    a = inputs.ALPHA
    layers = [dict(k=L["k"], stride=L["stride"], pool=L["pool"], pad=L.get("pad", "same")) for L in wl["layers"]]
    ws = [to_np(l["w"]) for l in st.L]
    bs = [to_np(l["b"]) for l in st.L]
    acts = oracle.stack_forward(to_np(st.x), layers, ws, bs, a)
    for i, l in enumerate(st.L):
        out = l["p"] if l["spec"]["pool"] else l["z"]
        e = maxabs_err(to_np(out), acts[i]["out"])
        assert e <= TOL["f32"], (i, e)
    # backward, op by op, from the GPU's own tensors
    g = dout
    for i in range(len(st.L) - 1, -1, -1):
        l = st.L[i]
        s = l["spec"]
        xin = to_np(st.layer_input(i))
        if l["fused"]:
            dz = fused_dz(l, g, a)
            dbr = dz.reshape(-1, s["cout"]).sum(0)
        elif l["fused_y"]:
            # weight and data gradients formed dz from (dy, y) themselves
            dz, dbr = oracle.bias_lrelu_bwd(to_np(g), to_np(l["z"]), a)
        else:
            dy = oracle.avgpool3d_bwd(to_np(g), l["out_dhw"]) if s["pool"] else to_np(g)
            if s["pool"]:
                e = maxabs_err(to_np(l["dy"]), dy)
                assert e <= TOL["f32"], ("pool_bwd", i, e)
            dzr, dbr = oracle.bias_lrelu_bwd(to_np(l["dy"] if s["pool"] else g), to_np(l["z"]), a)
            e = maxabs_err(to_np(l["dz"]), dzr)
            assert e <= TOL["f32"], ("lrelu_bwd", i, e)
            dz = to_np(l["dz"])
        e = maxabs_err(to_np(l["db"]), dbr)
        assert e <= TOL["f32"], ("db", i, e)
        pad = s.get("pad", "same")
        dwr = oracle.conv3d_bwd_weight(xin, dz, s["k"], stride=s["stride"], pad=pad)
        e = maxabs_err(to_np(l["dw"]), dwr)
        assert e <= TOL["f32"], ("wgrad", i, e)
        if l["dx"] is not None:
            dxr = oracle.conv3d_bwd_data(dz, to_np(l["w"]), l["in_dhw"], stride=s["stride"], pad=pad)
            e = maxabs_err(to_np(l["dx"]), dxr)
            assert e <= TOL["f32"], ("dgrad", i, e)
            g = l["dx"]


def sample_idx(rng, shape, n):
    return np.stack([rng.integers(0, t, n) for t in shape], 1)


def with_argmax(idx, t):
    """idx plus the index of the largest |value| of the GPU tensor t, so that the
    element that dominates the tensor is itself checked against the oracle."""
    a = np.unravel_index(int(np.argmax(np.abs(t))), t.shape)
    return np.concatenate([idx, np.asarray(a, dtype=idx.dtype)[None]], 0)


def sampled_err(got, ref):
    """max|gpu - oracle| over the sample / max|oracle| over the sample: the gate's
    scale comes from the oracle, never from the tensor under test."""
    return maxabs_err(np.asarray(got), np.asarray(ref))


def check_mask_points(l, xin, w, b, pts, stride, pad):
    """The fused forward's slope-mask bits at conv-output points pts[:, (n,d,h,w,c)]
    against the oracle's sign of u = z + b, wherever fp32 and fp64 cannot round
    u to different signs (|u| above a small fraction of the sample's max |u|)."""
    u = oracle.conv3d_fwd_points(xin, w, pts, stride=stride, pad=pad) + b[pts[:, 4]]
    bits = mask_bits(l)[tuple(pts.T)]
    decided = np.abs(u) > 1e-5 * np.abs(u).max()
    assert decided.mean() > 0.9
    bad = np.nonzero(bits[decided] != (u > 0)[decided])[0]
    assert bad.size == 0, ("mask", pts[decided][bad[:5]], u[decided][bad[:5]])


FULL = [("layer1_32c", True, False), ("stack_128c_b1_f32", True, False), ("stack_128c_b8_bf16", True, False),
        ("stack_128c_b8_bf16", True, True), ("stack_128c_b8_bf16", False, False),
        ("paper_c1c3_128_b8_bf16", True, False), ("paper_c1c3_128_b1_f32", True, False),
        ("stack_256c4_b2_bf16", True, False)]


@pytest.mark.parametrize("name,fused,rand_bias", FULL,
                         ids=["-".join([n, "fused" if f else "unfused"] + (["bias"] if r else [])) for n, f, r in FULL])
def test_full_size_sampled(name, fused, rand_bias):
    """At the workloads' full sizes, in the launch configuration the benchmark
    times (fused) and through the unfused entry points.  rand_bias: biases
    drawn from N(0, 0.1^2) instead of the timed workloads' zeros, so the bias
    paths of every kernel run with non-zero values at full size."""
    wl, st, dout = build(name, fused=fused)
    if rand_bias:
        ws, _ = inputs.make_weights(name)
        brng = np.random.default_rng(4242)
        st.set_params(ws, [brng.standard_normal(L["cout"]) * 0.1 for L in wl["layers"]])
    st.forward()
    st.backward(dout)
    torch.cuda.synchronize()
    dt = wl["dtype"]
    a = inputs.ALPHA
    rng = np.random.default_rng(99)
    ns = 96
    g = dout
    # forward, per layer: y (or pooled y) at sampled points from the layer's own input
    for i, l in enumerate(st.L):
        s = l["spec"]
        pad = s.get("pad", "same")
        xin = to_np(st.layer_input(i))
        w = to_np(l["w"])
        b = to_np(l["b"])
        if l["fused"]:
            pgpu = to_np(l["p"])
            pidx = with_argmax(sample_idx(rng, l["p"].shape, ns), pgpu)
            ref, win = [], []
            for n, pd, ph, pw, c in pidx:
                pts = [(n, 2 * pd + u, 2 * ph + v, 2 * pw + t, c) for u in (0, 1) for v in (0, 1) for t in (0, 1)]
                win += pts
                zz = oracle.conv3d_fwd_points(xin, w, pts, stride=s["stride"], pad=pad) + b[c]
                ref.append(np.mean(np.where(zz > 0, zz, a * zz)))
            e = sampled_err(pgpu[tuple(pidx.T)], ref)
            assert e <= TOL[dt], ("fwd", i, e)
            # the mask the backward pass consumes: every element of the sampled
            # windows, plus conv-output points drawn over the whole tensor (the
            # persistent kernels' later tiles included)
            mpts = np.concatenate([np.asarray(win), sample_idx(rng, (st.batch,) + l["out_dhw"] + (s["cout"],), 1024)])
            check_mask_points(l, xin, w, b, mpts, s["stride"], pad)
        else:
            zgpu = to_np(l["z"])
            zidx = with_argmax(sample_idx(rng, l["z"].shape, ns), zgpu)
            zz = oracle.conv3d_fwd_points(xin, w, zidx, stride=s["stride"], pad=pad) + b[zidx[:, 4]]
            ref = np.where(zz > 0, zz, a * zz)
            e = sampled_err(zgpu[tuple(zidx.T)], ref)
            assert e <= TOL[dt], ("fwd", i, e)
    # backward, per layer, teacher-forced from the GPU's dz (or g + mask)
    for i in range(len(st.L) - 1, -1, -1):
        l = st.L[i]
        s = l["spec"]
        pad = s.get("pad", "same")
        xin = to_np(st.layer_input(i))
        if l["fused"]:
            dz = fused_dz(l, g, a)
        elif l["fused_y"]:
            dz = oracle.bias_lrelu_bwd(to_np(g), to_np(l["z"]), a)[0]
        else:
            dz = to_np(l["dz"])
        dwg = to_np(l["dw"])
        widx = with_argmax(sample_idx(rng, l["dw"].shape, 64), dwg)
        ref = oracle.conv3d_bwd_weight_points(xin, dz, s["k"], widx, stride=s["stride"], pad=pad)
        e = sampled_err(dwg[tuple(widx.T)], ref)
        assert e <= TOL[dt], ("wgrad", i, e)
        dbr = dz.reshape(-1, s["cout"]).sum(0)
        e = maxabs_err(to_np(l["db"]), dbr)
        assert e <= TOL[dt], ("db", i, e)
        if l["dx"] is not None:
            dxg = to_np(l["dx"])
            xidx = with_argmax(sample_idx(rng, l["dx"].shape, ns), dxg)
            ref = oracle.conv3d_bwd_data_points(dz, to_np(l["w"]), l["in_dhw"], xidx, stride=s["stride"], pad=pad)
            e = sampled_err(dxg[tuple(xidx.T)], ref)
            assert e <= TOL[dt], ("dgrad", i, e)
            g = l["dx"]


@pytest.mark.parametrize("name", ["stack_128c_b8_bf16", "stack_64c_b1_f32"])
def test_two_stream_backward_is_bitwise_identical(name):
    """The deep layers' weight gradients on a second stream give the same bits
    as the single-stream step (every kernel's result is independent of what
    runs beside it), over two steps in a row."""
    wl = inputs.WORKLOADS[name]
    ws, bs = inputs.make_weights(name)
    x = inputs.make_input(name)
    outs = []
    for overlap in (True, False):
        st = ConvStack(wl["layers"], wl["size"], wl["batch"], wl["dtype"], inputs.ALPHA, "cuda", overlap_wgrad=overlap)
        st.set_params(ws, bs)
        st.set_input(x)
        dout = torch.as_tensor(inputs.normal((wl["batch"],) + st.out_dhw + (wl["layers"][-1]["cout"],),
                                             30000 + wl["cfg"]), device="cuda").to(st.tdt)
        for _ in range(2):
            st.forward()
            st.backward(dout)
        torch.cuda.synchronize()
        outs.append([(l["dw"].clone(), l["db"].clone(), None if l["dx"] is None else l["dx"].clone()) for l in st.L])
        del st
    for (a_dw, a_db, a_dx), (b_dw, b_db, b_dx) in zip(*outs):
        assert torch.equal(a_dw, b_dw) and torch.equal(a_db, b_db)
        assert (a_dx is None and b_dx is None) or torch.equal(a_dx, b_dx)
