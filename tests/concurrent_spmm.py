"""Run by tests/test_concurrency.py in a fresh process, so that the library's
launch-shape caches start empty: 8 host threads, each on its own HIP stream,
call nmg_spmm at the same moment on one layer, and every result must equal a
later single-thread call bit for bit.  The layers are the 768 x 768 x 128
single linear (2:4:4, the gathering kernel with its k-split across the waves
of a workgroup, whose split count comes from the cached occupancy figures)
and the 768 x 3072 x 4096 FFN down-projection (1:10:16)."""
import sys
import threading

import torch

from paper_2304_07613_amd import nmg, synth

THREADS = 8


def run(workload: int, kernel: str) -> None:
    lin = synth.WORKLOADS[workload].layers[0]
    W, X = synth.layer_inputs(workload, 0, lin)
    W, X = W.to("cuda:0"), X.to("cuda:0")
    v, idx, L = nmg.compress(W, lin.n, lin.m, lin.g)
    streams = [torch.cuda.Stream() for _ in range(THREADS)]
    Ys = [torch.full((L.M, lin.N), float("nan"), device="cuda:0") for _ in range(THREADS)]
    torch.cuda.synchronize()
    barrier = threading.Barrier(THREADS)
    errors = []

    def work(i: int) -> None:
        try:
            with torch.cuda.stream(streams[i]):
                barrier.wait()
                nmg.spmm_into(L, v, idx, X, Ys[i], kernel)
        except BaseException as e:  # reported by the main thread
            errors.append(e)

    threads = [threading.Thread(target=work, args=(i,)) for i in range(THREADS)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    if errors:
        raise errors[0]
    ref = nmg.spmm(v, idx, X, L, kernel)
    torch.cuda.synchronize()
    for i, Y in enumerate(Ys):
        same = torch.equal(Y.view(torch.int32), ref.view(torch.int32))
        print(f"workload {workload} kernel {kernel} thread {i}: "
              f"{'identical' if same else 'DIFFERENT'}", flush=True)
        if not same:
            sys.exit(1)


if __name__ == "__main__":
    nmg.lib()
    run(1, "mfma_direct")
    run(3, "auto")
    print("all identical", flush=True)
