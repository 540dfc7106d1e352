"""Element-by-element comparison of the GPU library's output with the oracle.

Bars: structure (row pointers, column ids) bit-exact; int32 counts and
Jaccard values bit-exact; fp64 values within 1e-12 and fp32 values within
1e-5 relative to the sum of |terms| of the entry (equal to |value| for the
non-negative workloads).
"""
import numpy as np

TOL = {"f64": 1e-12, "f32": 1e-5}


def device_rows(C, rows):
    """(row_ptr_of_subset, col, val) of the listed rows of a DeviceCSR, copying
    only those rows to the host."""
    import torch
    rp = C.row_ptr.cpu().numpy()
    rows = np.asarray(rows, dtype=np.int64)
    starts, ends = rp[rows], rp[rows + 1]
    lens = ends - starts
    sub_rp = np.zeros(len(rows) + 1, dtype=np.int64)
    np.cumsum(lens, out=sub_rp[1:])
    idx = np.repeat(starts - sub_rp[:-1], lens) + np.arange(sub_rp[-1])
    it = torch.from_numpy(idx).to(C.col_idx.device)
    col = C.col_idx[it].cpu().numpy() if len(idx) else np.zeros(0, np.int32)
    val = None
    if C.values is not None:
        val = C.values[it].cpu().numpy() if len(idx) else np.zeros(0, C.values.cpu().numpy().dtype)
    return sub_rp, col, val


def assert_match(gpu_rp, gpu_col, gpu_val, ref, semiring, what=""):
    np.testing.assert_array_equal(gpu_rp, ref.row_ptr, err_msg=f"{what}: row_ptr")
    np.testing.assert_array_equal(gpu_col, ref.col_idx, err_msg=f"{what}: col_idx")
    if semiring in ("count",):
        np.testing.assert_array_equal(gpu_val, ref.values, err_msg=f"{what}: counts")
    elif semiring == "jaccard":
        np.testing.assert_array_equal(gpu_val.view(np.uint32), ref.values.astype(np.float32).view(np.uint32),
                                      err_msg=f"{what}: jaccard bits")
    elif semiring in TOL:
        g = gpu_val.astype(np.float64)
        r = ref.values.astype(np.float64)
        scale = ref.sum_abs if ref.sum_abs is not None else np.abs(r)
        err = np.abs(g - r)
        bad = err > TOL[semiring] * scale
        if bad.any():
            k = int(np.flatnonzero(bad)[0])
            raise AssertionError(f"{what}: {int(bad.sum())} values out of tolerance; first at {k}: "
                                 f"gpu {g[k]!r} oracle {r[k]!r} scale {scale[k]!r}")
    else:
        raise ValueError(semiring)


def compare_full(C, ref, semiring, what=""):
    rp, col, val = C.to_host()
    assert C.nnz == ref.nnz, f"{what}: nnz {C.nnz} != {ref.nnz}"
    assert_match(rp, col, val, ref, semiring, what)


def compare_rows(C, ref, rows, semiring, what=""):
    rp, col, val = device_rows(C, rows)
    assert_match(rp, col, val, ref, semiring, what)
