"""DGC's sparsity warm-up (DGC is the paper's sparsification operator,
Sec. 5.1): a host-side schedule of the compression ratio over the first
epochs of training.  The ratio is an argument of every compress call, so
the schedule needs no device state; momentum correction and masking are
bytecomp_compress_dgc in the C library (binding.DgcCall)."""


def warmup_ratio(epoch: int, final_ratio: float, warmup_epochs: int = 4) -> float:
    """Density kept at `epoch`: it falls by a factor of four per warm-up
    epoch from 25% (sparsity 75%, 93.75%, 98.4375%, 99.6%, as in DGC's
    schedule), never below `final_ratio`, and is `final_ratio` from
    `warmup_epochs` on."""
    if epoch >= warmup_epochs:
        return float(final_ratio)
    return float(max(final_ratio, 0.25 ** (epoch + 1)))
