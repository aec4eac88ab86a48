"""Benchmark of the ResNet-18 training step on one MI355X (first version)."""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the training step runs on one GPU and no multi-GPU path is built",
              file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch
    from paper_2509_26092_amd import binding as B
    from paper_2509_26092_amd import inputs
    res = []
    for arch, classes, prec, N, H in [("cifar", 100, "fp32", 128, 32), ("imagenet", 1000, "bf16", 256, 224)]:
        w = B.Worker(arch, classes, prec)
        st = torch.zeros(w.n_state, device="cuda")
        ctx2 = B.rn18_init(w.cfg, 1, st)
        B.rn18_destroy(ctx2)
        x = torch.from_numpy(inputs.images(1, N, H, H)).cuda()
        y = torch.from_numpy(inputs.labels(1, N, classes)).cuda()
        loss = torch.zeros(1, device="cuda")
        for _ in range(args.warmup):
            w.train_step(st, x, y, 0.01, loss)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            w.train_step(st, x, y, 0.01, loss)
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / args.steps
        print("%s %s N=%d H=%d: %.2f ms/step, %.0f img/s, loss %.4f status %d" %
              (arch, prec, N, H, dt * 1e3, N / dt, loss.item(), w.sync_status()), flush=True)
        w.close()


if __name__ == "__main__":
    main()
