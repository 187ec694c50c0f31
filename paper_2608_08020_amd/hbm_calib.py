"""Plain device-to-device copy of a known size, for scaling HBM counters.

Run under `rocprofv3 --pmc FETCH_SIZE` (then WRITE_SIZE): each copy kernel
reads and writes exactly COPY_BYTES, so counter / COPY_BYTES is the factor
that turns the counter of another kernel into bytes.
"""
import torch

COPY_BYTES = 1 << 30
REPEATS = 4

if __name__ == "__main__":
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(REPEATS):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(f"copied {REPEATS} x {COPY_BYTES} bytes", flush=True)
