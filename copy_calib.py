"""Plain device-to-device copy of a known size, for calibrating memory counters.

Runs ``torch``'s copy kernel over a 1 GiB fp32 buffer a few times. Profiling it with
the same counters as a kernel of interest (FETCH_SIZE, WRITE_SIZE) gives the ratio
between counter readings and the bytes actually moved (1 GiB read and 1 GiB written
per dispatch).

    python copy_calib.py
"""
import torch

NBYTES = 1 << 30


def main() -> None:
    n = NBYTES // 4
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    print(f"copied {NBYTES} bytes x 3", flush=True)


if __name__ == "__main__":
    main()
