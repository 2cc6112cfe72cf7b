"""Calls from several host threads at once, each on its own stream: the
library's shared host state (the pinned staging ring of descriptor tables,
the per-device GEMM handle and plans, the per-thread error code) must keep
every call's result identical, bit for bit, to the same call made alone.
Routes: the fused map (T = 32), the GEMM-path map (T = 64), and the
optimizer step inside the fused kernel (T = 128) and on the GEMM path
(T = 512), each thread with its own weights and momenta."""
import threading

import pytest

import paper_2606_27216_amd as hm
import workloads

pytestmark = pytest.mark.gpu


def _batch(seed, dev):
    # 40 matrices: more than the 32 whose tables ride in the launch arguments,
    # so every fused call stages its table through the pinned ring
    shapes = [(96 + 32 * (i % 5), 64 + 32 * (i % 3)) for i in range(40)]
    return [workloads.gaussian(h, w, seed + i, "bf16", dev) for i, (h, w) in enumerate(shapes)]


@pytest.mark.parametrize("route", ["fused", "gemm"])
def test_threads_on_their_own_streams_match_single_calls(route):
    import torch
    dev = torch.device("cuda:0")
    print(f"[gpu-case] concurrency {route}", flush=True)
    n_threads, reps = 4, 6
    batches = [_batch(900 + 100 * t, dev) for t in range(n_threads)]

    def call(mats, stream):
        if route == "fused":
            return hm.ns_tiled(mats, T=32, K=5, stream=stream)
        return hm.ns_gemm(mats, T=64, K=5, stream=stream)

    torch.cuda.synchronize()
    ref = []
    for mats in batches:  # alone, one after the other, on the current stream
        ref.append([y.clone() for y in call(mats, torch.cuda.current_stream(dev))])
    torch.cuda.synchronize()

    results = [None] * n_threads
    errors = []

    def worker(t):
        try:
            torch.cuda.set_device(dev)
            s = torch.cuda.Stream(device=dev)
            outs = None
            with torch.cuda.stream(s):
                for _ in range(reps):
                    outs = call(batches[t], s)
            s.synchronize()
            results[t] = outs
        except Exception as e:  # reported below, on the test's thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(n_threads)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    assert not errors, errors
    for t in range(n_threads):
        for y, r in zip(results[t], ref[t]):
            assert torch.equal(y, r)


@pytest.mark.parametrize("T", [128, 512])
def test_threads_step_on_their_own_streams_match_single_calls(T):
    import torch
    dev = torch.device("cuda:0")
    print(f"[gpu-case] concurrency step T={T}", flush=True)
    n_threads, reps = 4, 3
    shapes = [(160 + 32 * (i % 5), 192 + 64 * (i % 3)) for i in range(36)]
    grads = [[workloads.gaussian(h, w, 5000 + 100 * t + i, "bf16", dev) for i, (h, w) in enumerate(shapes)]
             for t in range(n_threads)]
    w0 = [[workloads.gaussian(h, w, 7000 + 100 * t + i, "bf16", dev) for i, (h, w) in enumerate(shapes)]
          for t in range(n_threads)]

    def run(t, stream):
        ws = [x.clone() for x in w0[t]]
        ms = [torch.zeros_like(x) for x in w0[t]]
        for _ in range(reps):
            hm.step(ws, grads[t], ms, T=T, K=5, lr=0.02, weight_decay=0.1, stream=stream)
        return ws, ms

    torch.cuda.synchronize()
    ref = [run(t, torch.cuda.current_stream(dev)) for t in range(n_threads)]
    torch.cuda.synchronize()

    results = [None] * n_threads
    errors = []

    def worker(t):
        try:
            torch.cuda.set_device(dev)
            s = torch.cuda.Stream(device=dev)
            with torch.cuda.stream(s):
                results[t] = run(t, s)
            s.synchronize()
        except Exception as e:  # reported below, on the test's thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(n_threads)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    assert not errors, errors
    for t in range(n_threads):
        for y, r in zip(results[t][0] + results[t][1], ref[t][0] + ref[t][1]):
            assert torch.equal(y, r)
