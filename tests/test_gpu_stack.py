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


@pytest.mark.parametrize("name,fused", [("layer1_32c", True), ("stack_128c_b1_f32", True), ("stack_128c_b8_bf16", True),
                                        ("stack_128c_b8_bf16", False), ("paper_c1c3_128_b8_bf16", True),
                                        ("stack_256c4_b2_bf16", True)])
def test_full_size_sampled(name, fused):
    """At the workloads' full sizes, in the launch configuration the benchmark
    times (fused) and through the unfused entry points."""
    wl, st, dout = build(name, fused=fused)
    st.forward()
    st.backward(dout)
    torch.cuda.synchronize()
    dt = wl["dtype"]
    a = inputs.ALPHA
    rng = np.random.default_rng(99)
    ns = 48
    g = dout
    # forward, per layer: y (or pooled y) at sampled points from the layer's own input
    for i, l in enumerate(st.L):
        s = l["spec"]
        xin = to_np(st.layer_input(i))
        w = to_np(l["w"])
        b = to_np(l["b"])
        if l["fused"]:
            pidx = sample_idx(rng, l["p"].shape, ns)
            ref = []
            for n, pd, ph, pw, c in pidx:
                pts = [(n, 2 * pd + u, 2 * ph + v, 2 * pw + t, c) for u in (0, 1) for v in (0, 1) for t in (0, 1)]
                zz = oracle.conv3d_fwd_points(xin, w, pts, stride=s["stride"], pad=s.get("pad", "same")) + b[c]
                ref.append(np.mean(np.where(zz > 0, zz, a * zz)))
            got = to_np(l["p"])[tuple(pidx.T)]
        else:
            zidx = sample_idx(rng, l["z"].shape, ns)
            zz = oracle.conv3d_fwd_points(xin, w, zidx, stride=s["stride"], pad=s.get("pad", "same")) + b[zidx[:, 4]]
            ref = np.where(zz > 0, zz, a * zz)
            got = to_np(l["z"])[tuple(zidx.T)]
        e = maxabs_err(got, np.asarray(ref))
        assert e <= TOL[dt], ("fwd", i, e)
    # backward, per layer, teacher-forced from the GPU's dz (or g + mask)
    for i in range(len(st.L) - 1, -1, -1):
        l = st.L[i]
        s = l["spec"]
        xin = to_np(st.layer_input(i))
        dz = fused_dz(l, g, a) if l["fused"] else to_np(l["dz"])
        widx = sample_idx(rng, l["dw"].shape, 24)
        ref = oracle.conv3d_bwd_weight_points(xin, dz, s["k"], widx, stride=s["stride"], pad=s.get("pad", "same"))
        e = maxabs_err(to_np(l["dw"])[tuple(widx.T)], ref)
        # a sample of dW: normalise by the largest |dW| of the full GPU tensor
        scale = np.abs(to_np(l["dw"])).max()
        assert np.abs(to_np(l["dw"])[tuple(widx.T)] - ref).max() <= TOL[dt] * scale, ("wgrad", i, e)
        dbr = dz.reshape(-1, s["cout"]).sum(0)
        e = maxabs_err(to_np(l["db"]), dbr)
        assert e <= TOL[dt], ("db", i, e)
        if l["dx"] is not None:
            xidx = sample_idx(rng, l["dx"].shape, ns)
            ref = oracle.conv3d_bwd_data_points(dz, to_np(l["w"]), l["in_dhw"], xidx, stride=s["stride"],
                                                pad=s.get("pad", "same"))
            got = to_np(l["dx"])[tuple(xidx.T)]
            scale = np.abs(to_np(l["dx"])).max()
            assert np.abs(got - ref).max() <= TOL[dt] * scale, ("dgrad", i)
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
