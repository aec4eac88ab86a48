"""Maximum batch size from a linear memory model (Sec. 5.3, Eq. 9).

The paper models the device memory a training step needs at batch B as
M(B) = sum_l p_l + B * sum_l a_l: a batch-independent part (parameters,
gradients, optimizer state, buffers) plus a per-sample part (activations and
their gradients). It fits the two sums by linear regression over steps at
several batch sizes (64, 128, ..., 512), then takes the largest B with
M(B) <= M_GPU.

Here a "measurement" is the device memory in use (hipMemGetInfo) after one
training step of a fresh context minus the memory in use before it was
created: the context (momentum, weight shadows, workspace) and the caller's
state, images, labels and loss. This library adds a second bound besides the
memory: its kernels index each tensor with 32-bit offsets (convolutions are
launched over batch chunks to stay inside them), so a step is only planned
while every tensor stays below a fixed size; `addressing_max_batch` finds
that bound with the library's own planner (rn18_workspace_bytes returns 0
for a shape it rejects).
"""
import math

from . import planner


def fit(batches, used_bytes):
    """(sum p, sum a) of Eq. 9 by least squares over measured steps."""
    a, p = planner.fit_linear(batches, used_bytes)
    return p, a


def predict(p, a, batch):
    """M(B) of Eq. 9."""
    return p + a * batch


def max_batch(p, a, m_gpu):
    """The largest B with M(B) <= m_gpu (0 if not even one sample fits)."""
    if a <= 0:
        raise ValueError("the per-sample memory must be positive")
    b = math.floor((m_gpu - p) / a)
    while b > 0 and predict(p, a, b) > m_gpu:      # guard the floor against rounding
        b -= 1
    while predict(p, a, b + 1) <= m_gpu:
        b += 1
    return max(b, 0)


def addressing_max_batch(B, ctx, H, W, hi=1 << 20):
    """The largest N whose (N, H, W) step the library plans (bisection on
    rn18_workspace_bytes, a host-only query)."""
    def ok(n):
        return B.rn18_workspace_bytes(ctx, n, H, W) > 0
    if not ok(1):
        return 0
    lo = 1
    while hi - lo > 1:
        mid = (lo + hi) // 2
        if ok(mid):
            lo = mid
        else:
            hi = mid
    return lo


def measure_step(B, torch, arch, classes, prec, N, H, seed=1):
    """Device bytes in use by one training step of a fresh context at batch
    N and resolution H x H (images, labels, state, loss and the context),
    from hipMemGetInfo before and after; also the step's sticky status."""
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    free0, _ = torch.cuda.mem_get_info()
    n_state = B.rn18_state_floats(B.make_config(arch, classes, prec))[0]
    st = torch.zeros(n_state, device="cuda")
    w = B.Worker(arch, classes, prec, seed, state=st)
    try:
        g = torch.Generator(device="cuda")
        g.manual_seed(seed)
        x = torch.randn((N, 3, H, H), device="cuda", generator=g)
        y = torch.randint(0, classes, (N,), device="cuda", dtype=torch.int32, generator=g)
        loss = torch.zeros(1, device="cuda")
        w.train_step(st, x, y, 0.01, loss)
        status = w.sync_status()
        free1, _ = torch.cuda.mem_get_info()
        del x, y, loss
    finally:
        w.close()
        w.ws = None
        del st
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return free0 - free1, status


def profile(B, torch, arch, classes, prec, H, batches, seed=1):
    """Measured device bytes of a step at each batch size. A first step at
    the smallest batch is run and discarded: it loads the kernels' code and
    sets up the runtime's one-time state, which stays resident afterwards
    and is no part of any step's footprint."""
    measure_step(B, torch, arch, classes, prec, min(batches), H, seed)
    out = []
    for b in batches:
        used, status = measure_step(B, torch, arch, classes, prec, b, H, seed)
        if status != B.RN18_OK:
            raise B.Rn18Error(status, "training step at batch %d failed" % b)
        out.append(used)
    return out
