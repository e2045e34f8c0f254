"""Microbenchmark of the bf16 dense-layer kernel (rb_k_gemm_bf16).

Times Y = relu(X W^T + b) for the given M x N x K shapes through the C ABI,
with HIP events on torch's current stream, and prints TFLOP/s per shape. With
--ref it also times torch's own bf16 linear layer on the same operands (a
library GEMM with the bias fused and no activation, as a reference rate only).
Operands are seeded N(0, 1) inputs and N(0, 1/K) weights; outputs are not
checked here (the GPU tests do that).

    python3 -m paper_1712_06139_amd.gemm_bench --shapes 65536x8192x8192,32768x1024x1728 --ref
"""
from __future__ import annotations

import argparse

from . import rb


def main() -> None:
    import torch

    ap = argparse.ArgumentParser()
    ap.add_argument("--shapes", default="65536x8192x8192", help="comma list of MxNxK")
    ap.add_argument("--reps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--ref", action="store_true", help="also time torch's bf16 linear layer")
    args = ap.parse_args()
    if not torch.cuda.is_available():
        raise SystemExit("gemm_bench needs a GPU")
    lib = rb.lib()
    g = torch.Generator(device="cuda").manual_seed(0)
    for spec in args.shapes.split(","):
        M, N, K = (int(v) for v in spec.split("x"))
        X = torch.randn(M, K, device="cuda", generator=g).to(torch.bfloat16)
        W = (torch.randn(N, K, device="cuda", generator=g) / K ** 0.5).to(torch.bfloat16)
        b = torch.randn(N, device="cuda", generator=g) * 0.1
        b16 = b.to(torch.bfloat16)
        Y = torch.empty(M, N, device="cuda", dtype=torch.bfloat16)
        st = rb.torch_stream_ptr()

        def ours():
            rb.check(lib.rb_k_gemm_bf16(st, rb.dptr(X), K, rb.dptr(W), K, rb.dptr(b), rb.dptr(Y), N, M, N, K,
                                        rb.RB_ACT_RELU, 0), "rb_k_gemm_bf16")

        def ref():  # bias fused, no activation: the library GEMM alone
            torch.nn.functional.linear(X, W, b16)

        line = [f"{M}x{N}x{K}"]
        runs = (("rb_k_gemm_bf16", ours), ("torch_linear", ref)) if args.ref else (("rb_k_gemm_bf16", ours),)
        for name, fn in runs:
            for _ in range(args.warmup):
                fn()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(args.reps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / args.reps
            line.append(f"{name} {2.0 * M * N * K / us / 1e6:.0f} TFLOP/s ({us:.1f} us)")
        print("  ".join(line), flush=True)
        del X, W, b, b16, Y


if __name__ == "__main__":
    main()
