"""Records the small real MI355X trace sample that tests/golden/rocprof_sample
holds (run on a GPU machine; not part of the tests):

    rocprofv3 --kernel-trace --hip-runtime-trace --marker-trace --output-format csv \\
        -d OUT -o sample -- python3 tests/golden/capture_rocprof_trace.py

A few decode-like steps of a tiny MLP in PyTorch, each step and each layer
inside a named range (the CPU operators), eager launches, a synchronizing
copy back to the host per step, then the same step captured once as a HIP
graph and replayed (one launch API call per replay)."""
import ctypes

import torch


def _roctx():
    for name in ("librocprofiler-sdk-roctx.so", "libroctx64.so"):
        try:
            lib = ctypes.CDLL(name)
            lib.roctxRangePushA.argtypes = [ctypes.c_char_p]
            return lib
        except OSError:
            continue
    return None


RX = _roctx()


class Range:
    def __init__(self, name):
        self.name = name.encode()

    def __enter__(self):
        if RX:
            RX.roctxRangePushA(self.name)

    def __exit__(self, *exc):
        if RX:
            RX.roctxRangePop()


def main():
    torch.manual_seed(0)
    dev = "cuda"
    w1 = torch.randn(256, 512, device=dev)
    w2 = torch.randn(512, 256, device=dev)
    x = torch.randn(8, 256, device=dev)

    def step(x):
        with Range("layer1"):
            h = torch.relu(x @ w1)
        with Range("layer2"):
            y = torch.tanh(h @ w2)
        return y

    torch.cuda.synchronize()
    for s in range(6):
        with Range("decode_step"):
            y = step(x)
            with Range("sample"):
                v = float(y.sum().item())  # a synchronizing copy to the host
    # the same step as a captured graph, replayed
    static_x = x.clone()
    s_ = torch.cuda.Stream()
    s_.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s_):
        step(static_x)
    torch.cuda.current_stream().wait_stream(s_)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        static_y = step(static_x)
    for s in range(4):
        with Range("graph_step"):
            g.replay()
            with Range("sample"):
                v = float(static_y.sum().item())
    torch.cuda.synchronize()
    print("done", v)


if __name__ == "__main__":
    main()
