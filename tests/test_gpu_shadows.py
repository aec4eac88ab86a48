"""The per-step weight shadows: every conv's forward layout [Cout][KHW][Cin_p]
and data-gradient layout [Cin_p][KHW][Cout] hold exactly the storage-type
rounding of the fp32 state (zero in the padded input channels), for both
precisions and all three architectures. Expected values are plain reshapes
of the state: no oracle arithmetic is involved."""
import numpy as np
import pytest
import torch

from oracle import net
from paper_2509_26092_amd import binding as B
from paper_2509_26092_amd import inputs

pytestmark = pytest.mark.gpu


def storage_bits(x32, prec):
    t = torch.from_numpy(np.ascontiguousarray(x32, dtype=np.float32))
    if prec == "bf16":
        return t.to(torch.bfloat16).view(torch.int16).numpy()
    return t.view(torch.int32).numpy()


@pytest.mark.parametrize("arch,classes,prec,N,H", [("tiny", 10, "fp32", 2, 16), ("cifar", 100, "fp32", 2, 16),
                                                  ("cifar", 100, "bf16", 2, 16), ("imagenet", 1000, "bf16", 2, 64),
                                                  ("imagenet", 1000, "fp32", 2, 33)])
def test_weight_shadows_match_state(arch, classes, prec, N, H):
    L = net.Layout(arch, classes)
    w = B.Worker(arch, classes, prec)
    try:
        st = torch.zeros(w.n_state, device="cuda")
        B.rn18_destroy(B.rn18_init(w.cfg, 5, st))
        x = torch.from_numpy(inputs.images(5, N, H, H)).cuda()
        y = torch.from_numpy(inputs.labels(5, N, classes)).cuda()
        w.train_step(st, x, y, 0.0)          # lr 0: the state stays what the shadows were built from
        assert w.sync_status() == B.RN18_OK
        state = st.cpu().numpy()
        dt = torch.bfloat16 if prec == "bf16" else torch.float32
        itype = np.int16 if prec == "bf16" else np.int32
        for i, (name, cin, cout, k, s, p) in enumerate(L.convs):
            cin_p = cin if i > 0 else (4 if prec == "fp32" else 8)
            wt = L.get(state, name + ".w").reshape(cout, cin, k * k)
            full = np.zeros((cout, cin_p, k * k), np.float32)
            full[:, :cin] = wt
            want_f = storage_bits(full.transpose(0, 2, 1), prec)          # [Cout][KHW][Cin_p]
            got = torch.empty((cout, k * k, cin_p), dtype=dt, device="cuda")
            B.rn18_debug_copy(w.ctx, N, H, H, "wf", i, got)
            got_f = got.cpu().view(torch.int16 if prec == "bf16" else torch.int32).numpy().astype(itype)
            assert np.array_equal(got_f, want_f), (name, "forward layout")
            if i == 0:
                continue                      # the stem has no data gradient
            want_d = storage_bits(full.transpose(1, 2, 0), prec)          # [Cin_p][KHW][Cout]
            got = torch.empty((cin_p, k * k, cout), dtype=dt, device="cuda")
            B.rn18_debug_copy(w.ctx, N, H, H, "wd", i, got)
            got_d = got.cpu().view(torch.int16 if prec == "bf16" else torch.int32).numpy().astype(itype)
            assert np.array_equal(got_d, want_d), (name, "data-gradient layout")
    finally:
        w.close()
