#!/usr/bin/env python3
"""Per-iteration training time with SGD and with Jorge on one MI355X.

The analogue of the paper's per-iteration comparison (Table 1: ResNet-50 at a
batch of 1024 over 16 GPUs, i.e. 64 images per GPU, preconditioner updated
every 50 iterations): one data-parallel rank's iteration of ResNet-50 (v1.5,
random initialisation, channels-last, bf16 autocast) on synthetic 224 x 224
images with random labels: forward, backward and the optimizer step. SGD is
torch.optim.SGD (foreach) with momentum 0.9 and weight decay 5e-5; Jorge takes
its hyperparameters by single-shot tuning from those (Section 4) and runs
through JorgeOptimizer (one grouped library step for the 54 matrix weights,
heavy-ball SGD for the vectors). The gradient all-reduce of data-parallel
training is the same for every optimizer and is not part of this single-GPU
run. Prints one JSON line.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def resnet50(num_classes=1000):
    """ResNet-50 v1.5: stride on the 3x3 convolution of each bottleneck."""
    import torch.nn as nn

    class Bottleneck(nn.Module):
        def __init__(self, cin, width, stride):
            super().__init__()
            cout = 4 * width
            self.conv1 = nn.Conv2d(cin, width, 1, bias=False)
            self.bn1 = nn.BatchNorm2d(width)
            self.conv2 = nn.Conv2d(width, width, 3, stride, 1, bias=False)
            self.bn2 = nn.BatchNorm2d(width)
            self.conv3 = nn.Conv2d(width, cout, 1, bias=False)
            self.bn3 = nn.BatchNorm2d(cout)
            self.relu = nn.ReLU(inplace=True)
            self.down = None
            if stride != 1 or cin != cout:
                self.down = nn.Sequential(nn.Conv2d(cin, cout, 1, stride, bias=False), nn.BatchNorm2d(cout))

        def forward(self, x):
            idn = x if self.down is None else self.down(x)
            y = self.relu(self.bn1(self.conv1(x)))
            y = self.relu(self.bn2(self.conv2(y)))
            y = self.bn3(self.conv3(y))
            return self.relu(y + idn)

    layers = [nn.Conv2d(3, 64, 7, 2, 3, bias=False), nn.BatchNorm2d(64), nn.ReLU(inplace=True),
              nn.MaxPool2d(3, 2, 1)]
    cin = 64
    for width, blocks, stride in ((64, 3, 1), (128, 4, 2), (256, 6, 2), (512, 3, 2)):
        for b in range(blocks):
            layers.append(Bottleneck(cin, width, stride if b == 0 else 1))
            cin = 4 * width
    layers += [nn.AdaptiveAvgPool2d(1), nn.Flatten(), nn.Linear(cin, num_classes)]
    return nn.Sequential(*layers)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--batch", type=int, default=64, help="images per GPU per iteration")
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--intervals", default="50,1", help="Jorge preconditioner update intervals to time")
    ap.add_argument("--repeats", type=int, default=3,
                    help="rounds of (SGD, Jorge at each interval), interleaved in one process; medians reported")
    args = ap.parse_args()

    import torch
    import torch.nn.functional as F

    from paper_2310_12298_amd.optim import JorgeOptimizer, sgd_to_jorge

    torch.manual_seed(0)
    torch.cuda.set_device(0)
    # No exhaustive convolution-algorithm search: the same (default) kernels for every optimizer.
    torch.backends.cudnn.benchmark = False
    x = torch.randn(args.batch, 3, 224, 224, device="cuda").to(memory_format=torch.channels_last)
    y = torch.randint(0, 1000, (args.batch,), device="cuda")
    sgd_hp = dict(lr=0.1, momentum=0.9, weight_decay=5e-5)

    def say(*a):
        print(*a, file=sys.stderr, flush=True)

    def run(make_opt, name):
        torch.manual_seed(0)
        model = resnet50().cuda().to(memory_format=torch.channels_last)
        opt = make_opt(model)

        def it():
            opt.zero_grad(set_to_none=True)
            with torch.autocast("cuda", dtype=torch.bfloat16):
                loss = F.cross_entropy(model(x), y)
            loss.backward()
            opt.step()
            return loss

        for _ in range(args.warmup):
            it()
        torch.cuda.synchronize()
        say(f"{name}: warm-up done")
        t0 = time.perf_counter()
        for _ in range(args.steps):
            loss = it()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / args.steps
        say(f"{name}: {ms:.2f} ms per iteration")
        if not torch.isfinite(loss):
            raise RuntimeError("non-finite loss")
        n2d = sum(1 for p in model.parameters() if p.dim() >= 2)
        return ms, n2d

    out = {"metric": "ResNet-50 training iteration time (one data-parallel rank)", "unit": "ms/iteration",
           "batch_per_gpu": args.batch, "steps": args.steps, "warmup": args.warmup, "repeats": args.repeats,
           "dtype": "bf16 autocast", "data": "synthetic", "results": {}}
    jhp = sgd_to_jorge(sgd_hp["lr"], sgd_hp["momentum"], sgd_hp["weight_decay"])
    intervals = [int(v) for v in args.intervals.split(",") if v]
    runs = {"sgd": []}
    runs.update({f"jorge_k{k}": [] for k in intervals})
    n2d = None
    # Rounds interleave the optimizers, so drifts of the clock or of the box hit all of them alike.
    for r in range(args.repeats):
        runs["sgd"].append(run(lambda m: torch.optim.SGD(m.parameters(), foreach=True, **sgd_hp), f"sgd #{r}")[0])
        for k in intervals:
            ms, n2d = run(lambda m: JorgeOptimizer(m.parameters(), lr=jhp["lr"], beta1=jhp["beta1"],
                                                   weight_decay=jhp["weight_decay"],
                                                   vector_weight_decay=sgd_hp["weight_decay"],
                                                   precond_interval=k), f"jorge k={k} #{r}")
            runs[f"jorge_k{k}"].append(ms)
    med = {name: sorted(v)[len(v) // 2] for name, v in runs.items()}
    for name, v in runs.items():
        e = {"ms_per_iteration": med[name], "runs_ms": v, "images_per_s": args.batch / med[name] * 1e3}
        if name != "sgd":
            e["overhead_vs_sgd_pct"] = 100.0 * (med[name] - med["sgd"]) / med["sgd"]
            # per round, against that round's SGD run
            e["overhead_per_round_pct"] = [100.0 * (a - b) / b for a, b in zip(v, runs["sgd"])]
            e["matrix_params"] = n2d
        out["results"][name] = e
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
