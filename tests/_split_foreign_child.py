"""Child process of test_gpu_split_xcd.py: runs split-K GEMMs (slice-reduced
plans, streaming and tiled) and prints one line per case with the SHA-256 of
the output bytes.  NJ_TEST_SPLIT_FOREIGN (read once by the library) makes the
chunks in its bit mask behave as if dispatched to a foreign XCD."""
import hashlib
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import numpy as np  # noqa: E402
import torch  # noqa: E402

from paper_2512_22420_amd import binding as nb  # noqa: E402

CASES = [  # (kernel, split, M, N, K, epilogue)
    (nb.NJ_GEMM_STREAM, 8, 48, 4096, 4096, nb.NJ_GEMM_RESIDUAL),
    (nb.NJ_GEMM_STREAM, 4, 40, 6144, 4096, nb.NJ_GEMM_STORE),
    (nb.NJ_GEMM_STREAM, 2, 8, 2 * 2048, 2048, nb.NJ_GEMM_SWIGLU),
    (nb.NJ_GEMM_TILE_96x128, 2, 320, 4096, 4096, nb.NJ_GEMM_RESIDUAL),
    (nb.NJ_GEMM_TILE_160x256, 8, 320, 4096, 14336, nb.NJ_GEMM_RESIDUAL),
    (nb.NJ_GEMM_TILE_192x256, 4, 300, 2 * 1024, 4096, nb.NJ_GEMM_SWIGLU),
]


def main():
    torch.cuda.set_device(0)
    s = torch.cuda.current_stream().cuda_stream
    for kernel, split, M, N, K, epi in CASES:
        g = torch.Generator(device="cuda")
        g.manual_seed(M * 7 + N + K)
        Nout = N // 2 if epi == nb.NJ_GEMM_SWIGLU else N
        w_src = (torch.randn(N, K, device="cuda", generator=g) * 0.02).to(torch.bfloat16)
        w = torch.empty(nb.packed_weight_elems(N, K), dtype=torch.bfloat16, device="cuda")
        nb.pack_weight(w_src.data_ptr(), w.data_ptr(), N, K, s)
        x = torch.randn(M, K, device="cuda", generator=g).to(torch.bfloat16)
        tiled = kernel != nb.NJ_GEMM_STREAM
        xin = x.view(M, K // 32, 32).transpose(0, 1).contiguous() if tiled else x
        e = epi | (nb.NJ_GEMM_KBLOCKED if tiled else 0)
        y0 = torch.randn(M, Nout, device="cuda", generator=g)
        if epi == nb.NJ_GEMM_SWIGLU:
            y = torch.zeros((Nout // 32, M, 32) if tiled else (M, Nout), dtype=torch.bfloat16, device="cuda")
        else:
            y = torch.empty(M, Nout, device="cuda")
        nbytes = nb.gemm_plan_workspace_bytes(nb.NJ_BF16, M, N, K, e, kernel, split)
        ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        nb.workspace_init(ws.data_ptr(), nbytes, s)
        digests = []
        for rep in range(2):  # the second call runs on the counters the first left behind
            if epi != nb.NJ_GEMM_SWIGLU:
                y.copy_(y0)
            nb.gemm_with_plan(nb.NJ_BF16, xin.data_ptr(), w.data_ptr(), y.data_ptr(), M, N, K, e, kernel, split,
                              ws.data_ptr(), nbytes, s)
            torch.cuda.synchronize()
            out = y.cpu().view(torch.int16).numpy() if epi == nb.NJ_GEMM_SWIGLU else y.cpu().numpy()
            assert np.isfinite(out.astype(np.float32)).all() or epi == nb.NJ_GEMM_SWIGLU
            digests.append(hashlib.sha256(out.tobytes()).hexdigest()[:16])
        err = nb.device_error(ws.data_ptr(), nbytes, s)
        print(f"case kernel={kernel} split={split} M={M} N={N} K={K} epi={epi} err={err} "
              f"sha={digests[0]} repeat_same={digests[0] == digests[1]}", flush=True)


if __name__ == "__main__":
    main()
