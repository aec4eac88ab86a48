"""Helpers shared by the GPU parity tests: layout conversion between the
oracle's NCHW float64 arrays and the library's NHWC device tensors, the
parity metric, and a runner for one training step on either side."""
import numpy as np

from oracle import net, ops
from paper_2509_26092_amd import binding as B
from paper_2509_26092_amd import inputs

PREC = {"fp32": B.RN18_FP32, "bf16": B.RN18_BF16, "fp16": B.RN18_FP16}
# fp32 and the 16-bit mixed precisions (bf16, fp16 with loss scaling)
TOL = {"fp32": 1e-3, "bf16": 2e-2, "fp16": 2e-2}
HALF = ("bf16", "fp16")


def torch_dtype(prec):
    import torch
    return {"fp32": torch.float32, "bf16": torch.bfloat16, "fp16": torch.float16}[prec]


def to_dev_nhwc(x_nchw, prec, cpad=None):
    """float array [N,C,H,W] -> device NHWC tensor (channels zero-padded to cpad)."""
    import torch
    x = np.asarray(x_nchw, np.float32)
    if cpad and cpad > x.shape[1]:
        x = np.concatenate([x, np.zeros((x.shape[0], cpad - x.shape[1]) + x.shape[2:], np.float32)], axis=1)
    t = torch.from_numpy(np.ascontiguousarray(x.transpose(0, 2, 3, 1)))
    return t.to(torch_dtype(prec)).cuda().contiguous()


def from_dev_nhwc(t):
    return t.float().cpu().numpy().astype(np.float64).transpose(0, 3, 1, 2)


def rounded(x, prec):
    """What the device holds for an fp32 input in the given precision, as f64."""
    if prec == "bf16":
        return ops.round_bf16(x)
    if prec == "fp16":
        return ops.round_fp16(x)
    return np.asarray(x, np.float32).astype(np.float64)


def rel_errors(gpu, ref):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    d = gpu - ref
    nref = np.linalg.norm(ref)
    mref = np.abs(ref).max() if ref.size else 0.0
    rel = np.linalg.norm(d) / nref if nref > 0 else np.linalg.norm(d)
    mx = np.abs(d).max() / mref if mref > 0 else (np.abs(d).max() if d.size else 0.0)
    return rel, mx


def assert_close(gpu, ref, tol, name=""):
    """Parity metric: norm-wise relative error <= tol and, element by
    element, |gpu - ref| <= tol * max|ref| (a purely relative element bound
    is unbounded where ref crosses zero)."""
    rel, mx = rel_errors(gpu, ref)
    assert np.all(np.isfinite(gpu)), "%s: non-finite values" % name
    assert rel <= tol and mx <= tol, "%s: norm-rel %.3e, max-elem %.3e > tol %.1e" % (name, rel, mx, tol)
    return rel, mx


def make_state(arch, classes, seed):
    """Oracle-side initial state with every tensor kind non-trivial
    (random gamma, beta, FC bias and running statistics)."""
    L = net.Layout(arch, classes)
    st = net.init_state(L, seed)
    rng = np.random.default_rng(seed + 77)
    for name, cin, cout, k, s, p in L.convs:
        L.put(st, name + ".g", 1.0 + 0.1 * rng.standard_normal(cout))
        L.put(st, name + ".b", 0.1 * rng.standard_normal(cout))
        L.put(st, name + ".rm", 0.1 * rng.standard_normal(cout))
        L.put(st, name + ".rv", 1.0 + 0.1 * np.abs(rng.standard_normal(cout)))
    L.put(st, "fc.b", 0.1 * rng.standard_normal(classes))
    return L, st.astype(np.float32).astype(np.float64)


# Width of the band around a ReLU kink (|pre-activation| <= TAU * rms of the
# site) and around a max-pool tie (top-2 gap) inside which the choice of
# subgradient depends on the order of the fp32 sums that produced the value:
# the GPU's fp32 conv sums differ from exact ones by ~1e-6 relative. The
# same band serves bf16 steps, whose stored values the oracle mirrors
# exactly (see Mirror), so their kinks and ties are decided on the same
# values on both sides.
TAU = 1e-4


class Decider:
    """Decision rule for the oracle at non-unique points: keep the oracle's
    own ReLU mask / argmax everywhere, except at inputs the oracle itself
    finds within the rounding band, where the kernel's choice (read back
    from the stored activations) is taken if it is a valid one (a pool tap
    inside the image whose value is within the band of the window maximum).
    Counts how many choices were taken, how many in-band choices were
    invalid and how many GPU decisions outside the band disagree (both must
    be 0)."""

    def __init__(self, worker, N, H, prec, tau):
        self.w, self.N, self.H, self.prec, self.tau = worker, N, H, prec, tau
        self.ambiguous = 0
        self.taken = 0
        self.outside = 0
        self.invalid = 0
        self.sites = 0
        self.log = []

    def _fetch(self, which, index, shape_nchw, dtype=None):
        import torch
        n, c, h, w = shape_nchw
        dt = dtype or torch_dtype(self.prec)
        t = torch.empty((n, h, w, c), dtype=dt, device="cuda")
        B.rn18_debug_copy(self.w.ctx, self.N, self.H, self.H, which, index, t)
        torch.cuda.synchronize()
        return t.cpu().numpy().transpose(0, 3, 1, 2) if dt == torch.uint8 else from_dev_nhwc(t)

    def __call__(self, kind, site, pre, default):
        import torch
        self.sites += 1
        if kind == "relu":
            rms = np.sqrt(np.mean(pre * pre))
            amb = np.abs(pre) <= self.tau * rms
            if site == "stem":
                z = self._fetch("zstem", 0, pre.shape)
            else:
                z = self._fetch(site[0], site[1], pre.shape)
            gmask = z > 0
            ref = np.maximum(pre, 0.0)
            self.log.append((site, float(np.linalg.norm(z - ref) / max(np.linalg.norm(ref), 1e-300)),
                             int(((gmask != default) & ~amb).sum()), int(amb.sum())))
        else:
            x, arg = pre, default
            xp = np.pad(x, ((0, 0), (0, 0), (1, 1), (1, 1)), constant_values=-np.inf)
            ho, wo = arg.shape[2:]
            taps = np.stack([xp[:, :, kh:kh + 2 * (ho - 1) + 1:2, kw:kw + 2 * (wo - 1) + 1:2]
                             for kh in range(3) for kw in range(3)])
            top2 = -np.sort(-taps, axis=0)[:2]
            rms = np.sqrt(np.mean(x * x))
            amb = (top2[0] - top2[1]) <= self.tau * rms
            garg = self._fetch("parg", 0, arg.shape, torch.uint8).astype(np.int64)
            gmask = garg
            # a kernel's tap is acceptable only if it lies inside the image
            # and its value is within the band of the window's maximum
            tap = np.take_along_axis(taps, np.clip(garg, 0, 8)[None], axis=0)[0]
            valid = (garg >= 0) & (garg <= 8) & np.isfinite(tap) & (top2[0] - tap <= self.tau * rms)
            self.invalid += int((amb & ~valid).sum())
            amb = amb & valid
        self.ambiguous += int(amb.sum())
        self.outside += int(((gmask != default) & ~amb).sum())
        chosen = np.where(amb, gmask, default)
        self.taken += int((chosen != default).sum())
        return chosen


def tensor_shapes(L, N, H):
    """NCHW shapes of every rounding point / stored tensor of a step."""
    sh = {}
    name, cin, cout, k, s, p = L.convs[0]
    h = ops.conv_out_size(H, k, s, p)
    sh[("y", "stem")] = sh[("z", "stem")] = sh[("da_pool", 0)] = sh[("dy", "stem")] = (N, cout, h, h)
    c = cout
    if L.arch == "imagenet":
        h = ops.conv_out_size(h, 3, 2, 1)
    for bi, blk in enumerate(L.blocks):
        _, cin, cout, k, s, p = L.spec[blk["c1"]]
        ho = ops.conv_out_size(h, 3, s, 1)
        sh[("dx", bi)] = (N, cin, h, h)
        for cname in (blk["c1"], blk["c2"]) + ((blk["ds"],) if blk["ds"] else ()):
            sh[("y", cname)] = sh[("dy", cname)] = (N, cout, ho, ho)
        sh[("z", ("z1", bi))] = sh[("dz1", bi)] = sh[("z", ("out", bi))] = (N, cout, ho, ho)
        h, c = ho, cout
    sh[("da_avg", 0)] = (N, c, h, h)
    return sh


def _bf16_other_neighbor(exact, b):
    """The bf16 value on the other side of `exact` from its rounding b."""
    b32 = np.asarray(b, np.float32)
    u = b32.view(np.uint32).astype(np.int64)
    neg = (u >> 31) & 1
    up = exact > b
    inc_mag = np.where(up, neg == 0, neg == 1)
    un = np.where(inc_mag, u + 0x10000, u - 0x10000)
    un = np.where(b32 == 0, np.where(up, 0x00010000, 0x80010000), un)
    return un.astype(np.uint32).view(np.float32).astype(np.float64)


def _fp16_other_neighbor(exact, b):
    """The fp16 value on the other side of `exact` from its rounding b
    (b finite; the neighbour of the largest finite value is infinite)."""
    with np.errstate(over="ignore"):
        b16 = np.asarray(b, np.float64).astype(np.float16)
    u = b16.view(np.uint16).astype(np.int64)
    neg = (u >> 15) & 1
    up = exact > b
    inc_mag = np.where(up, neg == 0, neg == 1)
    un = np.where(inc_mag, u + 1, u - 1)
    un = np.where(b16 == 0, np.where(up, 0x0001, 0x8001), un)
    return un.astype(np.uint16).view(np.float16).astype(np.float64)


class Mirror(Decider):
    """Decider for 16-bit (bf16, fp16) steps that also mirrors the kernel's
    rounding decisions where they are not unique: a value whose exact (fp64)
    result lies within TAU_ROUND ulp (or TAU_ABS * rms) of a rounding
    midpoint may round either way in a kernel that computes it in fp32;
    there the kernel's stored value is taken, after checking it is one of
    the two neighbours in the 16-bit type. Everywhere else the kernel's
    stored value must equal the oracle's round-to-nearest-even result
    exactly. Backward tensors are captured from the kernel as they are
    produced (scaled by the loss scale in fp16 steps, on both sides)."""
    TAU_ROUND = 0.02
    TAU_ABS = 1e-5

    def __init__(self, worker, L, N, H, prec, tau):
        import torch
        super().__init__(worker, N, H, prec, tau)
        self.L = L
        self.shapes = tensor_shapes(L, N, H)
        self.conv_index = {c[0]: i for i, c in enumerate(L.convs)}
        self.cap = {}
        kinds = {"dy": "dy", "dz1": "dz1", "dx": "dx", "da_avg": "da_avg", "da_pool": "da_pool"}
        for (kind, idx), (n, c, h, w) in self.shapes.items():
            if kind not in kinds:
                continue
            if kind == "da_pool" and L.arch != "imagenet":
                continue
            index = self.conv_index[idx] if kind == "dy" else idx
            t = torch.full((n, h, w, c), float("nan"), dtype=torch_dtype(prec), device="cuda")
            B.rn18_debug_capture(worker.ctx, kind, index, t)
            self.cap[(kind, idx)] = t
        import time
        self.t0 = time.time()
        self.round_outside = 0
        self.round_invalid = 0
        self.round_taken = 0
        self.round_band = 0
        self.round_log = []

    def _gpu_value(self, point):
        kind, idx = point
        shape = self.shapes[point]
        if kind == "y":
            return self._fetch("y", self.conv_index[idx], shape)
        if kind == "z":
            if idx == "stem":
                return self._fetch("zstem", 0, shape)
            return self._fetch(idx[0], idx[1], shape)
        import torch
        torch.cuda.synchronize()
        return from_dev_nhwc(self.cap[point])

    def __call__(self, kind, site, pre, default):
        if self.N * self.H * self.H >= 1 << 22:
            # large comparisons take minutes: report each stored tensor as it is checked
            import time
            print("  %s %s  %.1f s" % (kind, site, time.time() - self.t0), flush=True)
        if kind != "round":
            return super().__call__(kind, site, pre, default)
        exact, b = pre, default
        g = self._gpu_value(site)
        nb = (_fp16_other_neighbor if self.prec == "fp16" else _bf16_other_neighbor)(exact, b)
        ulp = np.abs(nb - b)
        rms = np.sqrt(np.mean(exact * exact))
        band = np.abs(exact - 0.5 * (b + nb)) <= self.TAU_ROUND * ulp + self.TAU_ABS * rms
        # in the band the kernel may hold either neighbour, or (near zero,
        # where the absolute term dominates) any value that close to exact
        valid = (g == b) | (g == nb) | (np.abs(g - exact) <= 2 * self.TAU_ABS * rms)
        outside = (g != b) & ~band
        self.round_band += int(band.sum())
        self.round_outside += int(outside.sum())
        self.round_invalid += int((band & ~valid).sum())
        chosen = np.where(band & valid, g, b)
        self.round_taken += int((chosen != b).sum())
        if outside.any():
            i = np.argwhere(outside)[0]
            self.round_log.append((site, int(outside.sum()), tuple(int(v) for v in i), float(g[tuple(i)]),
                                   float(b[tuple(i)]), float(exact[tuple(i)])))
        return chosen

    def close(self):
        B.rn18_debug_capture(self.w.ctx, None, 0, None)


def gpu_train_step(arch, classes, prec, state64, x, y, lr, steps=1, momentum_in=None, worker=None):
    import torch
    w = worker or B.Worker(arch, classes, prec)
    st = torch.from_numpy(np.asarray(state64, np.float32)).cuda()
    xi = torch.from_numpy(np.asarray(x, np.float32)).cuda()
    yi = torch.from_numpy(np.asarray(y, np.int32)).cuda()
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    if momentum_in is not None:
        B.rn18_set_momentum(w.ctx, torch.from_numpy(np.asarray(momentum_in, np.float32)).cuda())
    losses = []
    for _ in range(steps):
        w.train_step(st, xi, yi, lr, loss)
        losses.append(float(loss.item()))
    v = torch.zeros(w.n_trainable, dtype=torch.float32, device="cuda")
    B.rn18_get_momentum(w.ctx, v)
    status = w.sync_status()
    out = st.cpu().numpy().astype(np.float64), v.cpu().numpy().astype(np.float64), losses, status
    if worker is None:
        w.close()
    return out


def compare_step(L, cfg, state0, x, y, lr, gpu_state, gpu_v, gpu_loss, tol, v0=None, decide=None):
    """Oracle train step from the same state; compare every tensor."""
    P = L.n_trainable
    v0 = np.zeros(P) if v0 is None else v0
    new, v1, loss, grad = net.train_step(cfg, L, state0, v0, x, y, lr, decide=decide)
    report = {}
    assert abs(gpu_loss - loss) <= tol * abs(loss), ("loss", gpu_loss, loss)
    for key in L.off:
        o, shp = L.off[key]
        n = int(np.prod(shp))
        if o < P:
            report[key + ".v"] = assert_close(gpu_v[o:o + n], v1[o:o + n], tol, key + " momentum (grad + wd*w)")
            report[key + ".dw"] = assert_close(state0[o:o + n] - gpu_state[o:o + n], state0[o:o + n] - new[o:o + n],
                                               tol, key + " update")
        report[key] = assert_close(gpu_state[o:o + n], new[o:o + n], tol, key)
    return report, loss
