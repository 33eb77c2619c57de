"""How the files in this folder were made (needs a GPU; not run by the tests).

A small CNN (two conv/batchnorm/ReLU blocks, pooling, a linear layer) trains
for four iterations with SGD; every layer's forward and backward pass and
every iteration sit in a marker range (torch.cuda.nvtx, which rocprofv3
records as roctx ranges).  Captured on one MI355X with

    rocprofv3 --kernel-trace --hip-runtime-trace --memory-copy-trace \\
        --marker-trace --output-format csv -d OUT -o run -- python3 capture.py

and then cut to the steady-state iterations 2 and 3 with `trim(OUT, here)`:
the calls that start inside those two iteration ranges, the kernels and
copies correlated with them, and the marker ranges that start inside; every
kept row is the line rocprofv3 wrote, unchanged.
"""
import csv
import os


def trim(src, dst, iterations=("iteration 2", "iteration 3"), prefix="run"):
    def rows(name):
        lines = open(os.path.join(src, "%s_%s.csv" % (prefix, name)), newline="").read()
        lines = lines.splitlines(keepends=True)
        hdr = next(csv.reader([lines[0]]))
        return lines[0], [(ln, dict(zip(hdr, next(csv.reader([ln]))))) for ln in lines[1:]]

    def write(name, head, kept):
        with open(os.path.join(dst, "%s_%s.csv" % (prefix, name)), "w", newline="") as f:
            f.write(head + "".join(ln for ln, _ in kept))

    mh, marks = rows("marker_api_trace")
    spans = [(int(r["Start_Timestamp"]), int(r["End_Timestamp"])) for _, r in marks
             if r["Function"].strip() in iterations]
    t0, t1 = min(a for a, _ in spans), max(b for _, b in spans)
    inside = lambda r: t0 <= int(r["Start_Timestamp"]) <= t1   # noqa: E731
    ah, api = rows("hip_api_trace")
    api = [x for x in api if inside(x[1])]
    corr = {int(r["Correlation_Id"]) for _, r in api}
    write("hip_api_trace", ah, api)
    for name in ("kernel_trace", "memory_copy_trace"):
        h, rs = rows(name)
        write(name, h, [x for x in rs if int(x[1]["Correlation_Id"]) in corr])
    write("marker_api_trace", mh, [x for x in marks if inside(x[1])])


def main():
    import torch
    import torch.nn as nn
    torch.manual_seed(0)
    dev = "cuda"
    model = nn.Sequential(
        nn.Conv2d(3, 16, 3, padding=1), nn.BatchNorm2d(16), nn.ReLU(),
        nn.Conv2d(16, 32, 3, padding=1), nn.BatchNorm2d(32), nn.ReLU(),
        nn.AdaptiveAvgPool2d(1), nn.Flatten(), nn.Linear(32, 10)).to(dev)
    opt = torch.optim.SGD(model.parameters(), lr=0.1, momentum=0.9)
    names = {m: "layer%d:%s" % (i, type(m).__name__) for i, m in enumerate(model)}

    def fpre(mod, inp):
        torch.cuda.nvtx.range_push("fwd " + names[mod])

    def fpost(mod, inp, out):
        torch.cuda.nvtx.range_pop()

    def bpre(mod, g):
        torch.cuda.nvtx.range_push("bwd " + names[mod])

    def bpost(mod, gi, go):
        torch.cuda.nvtx.range_pop()
    for m in model:
        m.register_forward_pre_hook(fpre)
        m.register_forward_hook(fpost)
        m.register_full_backward_pre_hook(bpre)
        m.register_full_backward_hook(bpost)
    x = torch.randn(8, 3, 16, 16)
    y = torch.randint(0, 10, (8,))
    for it in range(4):
        torch.cuda.nvtx.range_push("iteration %d" % it)
        xb, yb = x.to(dev), y.to(dev)
        loss = nn.functional.cross_entropy(model(xb), yb)
        opt.zero_grad()
        loss.backward()
        torch.cuda.nvtx.range_push("weight update")
        opt.step()
        torch.cuda.nvtx.range_pop()
        print("iteration", it, "loss", float(loss.item()), flush=True)
        torch.cuda.nvtx.range_pop()
    torch.cuda.synchronize()


if __name__ == "__main__":
    main()
