"""The fused step inside a real explicit-gradient inner loop (Listing 1): a
MAML-style meta-gradient through K inner Adam steps of a 4-block conv-net on
synthetic 28x28 one-channel, 5-way tasks, including the model's Hessian-vector
products.  The inner optimizer is MetaAdam (leaf-direct kernels through
AdamTreeFn); the reference is the same loop with torch.optim's functional Adam
(differentiable mode), in fp64 on the CPU and in fp32 on the GPU.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from workloads import HYPER

pytestmark = pytest.mark.gpu

LR, B1, B2, EPS = 1e-3, HYPER["b1"], HYPER["b2"], HYPER["eps"]


class ConvNet(torch.nn.Module):
    """4 x [conv3x3 (+ bias), BN (batch statistics) scale/shift, ReLU, 2x2 max-pool], linear.

    With conv_bias the biases sit in front of batch normalisation, which removes
    them: their gradient is zero in exact arithmetic and at rounding level in
    fp32 (some elements exactly zero), the 0/0 point of Adam's VJP and its
    neighbourhood."""

    def __init__(self, width=64, ways=5, conv_bias=True):
        super().__init__()
        c = 1
        self.conv_bias = conv_bias
        for i in range(4):
            self.register_parameter("w%d" % i, torch.nn.Parameter(torch.randn(width, c, 3, 3) * (2.0 / (9 * c)) ** 0.5))
            if conv_bias:
                self.register_parameter("b%d" % i, torch.nn.Parameter(torch.zeros(width)))
            self.register_parameter("s%d" % i, torch.nn.Parameter(torch.ones(width)))
            self.register_parameter("t%d" % i, torch.nn.Parameter(torch.zeros(width)))
            c = width
        self.head_w = torch.nn.Parameter(torch.randn(ways, width) * (1.0 / width) ** 0.5)
        self.head_b = torch.nn.Parameter(torch.zeros(ways))

    def forward(self, x):
        p = self._parameters
        for i in range(4):
            x = F.conv2d(x, p["w%d" % i], p["b%d" % i] if self.conv_bias else None, padding=1)
            x = F.batch_norm(x, None, None, p["s%d" % i], p["t%d" % i], training=True)
            x = F.max_pool2d(F.relu(x), 2)
        return F.linear(x.flatten(1), p["head_w"], p["head_b"])


def _task(seed, n=25):
    g = torch.Generator().manual_seed(seed)
    xs = torch.randn(n, 1, 28, 28, generator=g)
    ys = torch.arange(n) % 5
    xq = torch.randn(n, 1, 28, 28, generator=g)
    yq = torch.arange(n) % 5
    return xs, ys, xq, yq


def _meta_grad_ours(init, task, K, device, conv_bias=False, width=64):
    import paper_2211_06934_amd as P
    net = ConvNet(width=width, conv_bias=conv_bias).to(device)
    with torch.no_grad():
        for n, p in net.named_parameters():
            p.copy_(init[n])
    p0 = [p for _, p in net.named_parameters()]
    opt = P.MetaAdam(net, lr=LR, b1=B1, b2=B2, eps=EPS)
    xs, ys, xq, yq = (t.to(device) for t in task)
    for _ in range(K):
        opt.step(F.cross_entropy(net(xs), ys))
    outer = F.cross_entropy(net(xq), yq)
    return [g.detach().double().cpu() for g in torch.autograd.grad(outer, p0)], outer.item()


def _meta_grad_reference(init, task, K, device, dtype, conv_bias=False):
    from torch.optim.adam import adam
    net = ConvNet(conv_bias=conv_bias).to(device=device, dtype=dtype)
    names = [n for n, _ in net.named_parameters()]
    p0 = [init[n].to(device=device, dtype=dtype).clone().requires_grad_() for n in names]
    params = [p.clone() for p in p0]
    mu = [torch.zeros_like(p) for p in p0]
    nu = [torch.zeros_like(p) for p in p0]
    xs, ys, xq, yq = (t.to(device=device, dtype=dtype) if t.is_floating_point() else t.to(device) for t in task)

    def fwd(ps, x):
        for name, p in zip(names, ps):
            net._parameters[name] = p
        return net(x)

    for k in range(K):
        loss = F.cross_entropy(fwd(params, xs), ys)
        grads = list(torch.autograd.grad(loss, params, create_graph=True))
        params = [p.clone() for p in params]
        mu = [m.clone() for m in mu]
        nu = [v.clone() for v in nu]
        steps = [torch.tensor(float(k), dtype=dtype) for _ in params]
        adam(params, grads, mu, nu, [], steps, foreach=False, capturable=False, differentiable=True, fused=None,
             grad_scale=None, found_inf=None, has_complex=False, amsgrad=False, beta1=B1, beta2=B2, lr=LR,
             weight_decay=0.0, eps=EPS, maximize=False)
    outer = F.cross_entropy(fwd(params, xq), yq)
    return [g.detach().double().cpu() for g in torch.autograd.grad(outer, p0)], outer.item()


def _normrel(a, b):
    num = sum(float(torch.sum((x - y) ** 2)) for x, y in zip(a, b)) ** 0.5
    den = sum(float(torch.sum(y ** 2)) for y in b) ** 0.5
    return num / den


def torch32_spread(run_ref32, ref64, reps=3):
    """Largest distance from the fp64 loop over `reps` runs of torch's fp32
    loop on the GPU.  That loop is not deterministic (its convolution
    backward), and the meta-gradient is ill-conditioned enough that one run
    can land 1.8e-2 and the next 6.7e-2 from fp64 on identical inputs, so a
    single run is not a stable yardstick."""
    return max(_normrel(run_ref32(), ref64) for _ in range(reps))


@pytest.mark.parametrize("K", [1, 3])
def test_maml_meta_gradient_through_fused_adam(K):
    torch.manual_seed(0)
    init = {n: p.detach().clone() for n, p in ConvNet(conv_bias=False).named_parameters()}
    task = _task(5)
    ours, out_ours = _meta_grad_ours(init, task, K, "cuda")
    ref64, out64 = _meta_grad_reference(init, task, K, "cpu", torch.float64)
    ref32, out32 = _meta_grad_reference(init, task, K, "cuda", torch.float32)
    assert all(torch.isfinite(g).all() for g in ref64 + ref32)
    assert np.isfinite(out_ours) and abs(out_ours - out64) <= 1e-4 * abs(out64), (out_ours, out64)
    e32 = _normrel(ours, ref32)
    runs = [ours] + [_meta_grad_ours(init, task, K, "cuda")[0] for _ in range(2)]
    e64 = min(_normrel(r, ref64) for r in runs)
    t64 = torch32_spread(lambda: _meta_grad_reference(init, task, K, "cuda", torch.float32)[0], ref64)
    print("K=%d  |ours-torch32|=%.2e  min |ours-fp64|=%.2e  max |torch32-fp64|=%.2e" % (K, e32, e64, t64))
    # The meta-gradient of an Adam inner loop is ill-conditioned: the update
    # divides by |g|, so the fp32 model's rounding (conv, Hessian-vector
    # products) is amplified; both fp32 loops land ~1e-3 from fp64, and both
    # are nondeterministic through the convolution backward.  The bar here:
    # the nearest of three runs of ours is no further from the fp64 loop than
    # twice the farthest of three runs of torch's op-by-op fp32 loop (every
    # fused step of the loop is checked against the oracle element by element
    # in test_maml_fused_steps_match_oracle_inside_the_loop).
    assert e64 < 2e-2, e64
    assert e64 < 2 * t64 + 1e-5, (e64, t64)


def test_maml_zero_gradient_biases_stay_finite():
    # Conv biases in front of batch normalisation have a gradient that is zero
    # up to rounding, often exactly, so v' = 0 at step 1: the explicit 0/0
    # case of the fused VJP gives finite meta-gradients (an op-by-op sqrt
    # backward gives 0 * inf).
    torch.manual_seed(1)
    init = {n: p.detach().clone() for n, p in ConvNet(conv_bias=True).named_parameters()}
    ours, out_ours = _meta_grad_ours(init, _task(6), 2, "cuda", conv_bias=True)
    assert np.isfinite(out_ours)
    assert all(torch.isfinite(g).all() for g in ours)


def _recording_adam_tree_fn(log):
    """AdamTreeFn that also records, per call, what its kernels were given and
    what they returned: forward (count, p, g, m, v -> p', m', v') and backward
    (saved g, m, v and the incoming cotangents -> dp, dg, dm, dv), as fp64
    numpy arrays over the concatenated leaves."""
    import paper_2211_06934_amd as P
    base = P.autograd.AdamTreeFn
    cat = lambda ts: np.concatenate([t.detach().reshape(-1).double().cpu().numpy() for t in ts])  # noqa: E731

    class Rec(base):
        @staticmethod
        def forward(ctx, table, count, hyper, *leaves):
            out = base.forward(ctx, table, count, hyper, *leaves)
            S = len(leaves) // 4
            torch.cuda.synchronize()
            log.append(dict(kind="fwd", count=count, hyper=hyper,
                            inp=[cat(leaves[i * S:(i + 1) * S]) for i in range(4)],
                            out=[cat(out[i * S:(i + 1) * S]) for i in range(3)]))
            return out

        @staticmethod
        def backward(ctx, *cots):
            res = base.backward(ctx, *cots)
            S = ctx.S
            saved = ctx.saved_tensors
            torch.cuda.synchronize()
            zero_or = lambda grp, like: [torch.zeros_like(x) if c is None else c for c, x in zip(grp, like)]  # noqa
            log.append(dict(kind="bwd", count=ctx.count, hyper=ctx.hyper,
                            saved=[cat(saved[i * S:(i + 1) * S]) for i in range(3)],
                            cots=[cat(zero_or(cots[i * S:(i + 1) * S], saved[:S])) for i in range(3)],
                            res=[cat(res[3 + i * S:3 + (i + 1) * S]) for i in range(4)]))
            return res

    return Rec


@pytest.mark.parametrize("K,conv_bias,width", [(1, False, 64), (3, False, 64), (2, True, 64),
                                               (3, False, 16), (2, True, 16)])
def test_maml_fused_steps_match_oracle_inside_the_loop(K, conv_bias, width, monkeypatch):
    # Every fused step the real MAML loop runs -- warm moments after step 1,
    # cotangents that carry the model's Hessian-vector products into the
    # earlier steps, and (conv_bias) zero-gradient leaves at the 0/0 point
    # mixed with live ones -- checked element by element against the oracle
    # on the inputs that step actually received: 1e-5 of the term scale for
    # the forward, 1e-4 for the VJP, and the params cotangent passed through
    # bit for bit.  Width 64 (112,261 parameters) takes the tiled leaf-direct
    # kernels, width 16 (14 or 18 leaves, about 7,300 parameters) the
    # small-tree kernels.
    import oracle
    import paper_2211_06934_amd as P
    from tests.support import BWD_RTOL, FWD_RTOL, assert_mag_close
    log = []
    monkeypatch.setattr(P.autograd, "AdamTreeFn", _recording_adam_tree_fn(log))
    torch.manual_seed(2 + K)
    init = {n: p.detach().clone() for n, p in ConvNet(width=width, conv_bias=conv_bias).named_parameters()}
    grads, outer = _meta_grad_ours(init, _task(7 + K), K, "cuda", conv_bias=conv_bias, width=width)
    assert np.isfinite(outer) and all(torch.isfinite(g).all() for g in grads)
    fw = [r for r in log if r["kind"] == "fwd"]
    bw = [r for r in log if r["kind"] == "bwd"]
    assert [r["count"] for r in fw] == list(range(K)) and sorted(r["count"] for r in bw) == list(range(K))
    zero_g, tiny_g = 0, 0
    for r in fw:
        h = r["hyper"]
        hy = (r["count"], h.lr, h.b1, h.b2, h.eps, h.eps_root)
        p, g, m, v = r["inp"]
        ref = oracle.adam_fwd(p, g, m, v, *hy)
        mag = oracle.adam_fwd_mag(p, g, m, v, *hy)
        for name, got, x, mg in zip(("p'", "m'", "v'"), r["out"], ref, mag):
            assert_mag_close(got, x, mg, FWD_RTOL, "step %d %s" % (r["count"], name))
        zero_g += int(np.sum(g == 0.0))
        tiny_g += int(np.sum(np.abs(g) < 1e-8))  # s at or below eps: the neighbourhood of the 0/0 point
    for r in bw:
        h = r["hyper"]
        hy = (r["count"], h.lr, h.b1, h.b2, h.eps, h.eps_root)
        g, m, v = r["saved"]
        dP, dM, dV = r["cots"]
        ref = oracle.adam_bwd(dP, dM, dV, g, m, v, *hy)
        mag = oracle.adam_bwd_mag(dP, dM, dV, g, m, v, *hy)
        assert np.array_equal(r["res"][0], dP), "params cotangent is the identity"
        for name, got, x, mg in zip(("dg", "dm", "dv"), r["res"][1:], ref[1:], mag):
            assert_mag_close(got, x, mg, BWD_RTOL, "VJP step %d %s" % (r["count"], name))
    print("K=%d conv_bias=%s width=%d: %d gradient elements exactly 0, %d below 1e-8" % (K, conv_bias, width, zero_g,
                                                                                   tiny_g))
    if conv_bias:
        # the biases in front of batch normalisation have a gradient that is
        # zero in exact arithmetic and at rounding level in fp32: the loop
        # reaches the 0/0 point itself (exact zeros) and its neighbourhood
        assert tiny_g >= 1, (zero_g, tiny_g)
    # the cotangents of the earlier steps are not just the outer gradient:
    # they carry the model's second-order terms
    if K > 1:
        last = [r for r in bw if r["count"] == K - 1][0]
        first = [r for r in bw if r["count"] == 0][0]
        assert not np.allclose(first["cots"][0], last["cots"][0])
