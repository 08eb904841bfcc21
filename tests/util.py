"""Shared test helpers: moving bf16 bit patterns to and from the GPU, tolerances, and the
index-set rule for top-k comparisons."""
import numpy as np

# Tolerances of the GPU path against the fp64 oracle.
OUT_ATOL = 2e-2      # attention output, max abs (bf16 output)
LSE_ATOL = 1e-4      # log-sum-exp, abs
SAL_RTOL = 1e-3      # saliency, relative, every key
BAND = 1e-4          # relative band around the k-th largest oracle saliency


def out_error_bound(out_oracle, v_absmax):
    """Worst-case error of a bf16 attention output, with bf16's unit roundoff u = 2^-8:
    the probabilities are rounded to bf16 for the value product (relative error <= u
    each, so <= u max|v| after normalisation by the fp32 row sum); a split plan stores
    each partial output -- a convex combination of value rows -- in bf16 (<= u max|v|
    more, the merge weights summing to one); and the output is rounded to bf16
    (<= u |o|).  fp32 accumulation adds ~1e-6."""
    return 2.0 ** -8 * (float(np.abs(out_oracle).max()) + 2.0 * float(v_absmax)) + 1e-5


def to_dev(a):
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).cuda()
    return torch.from_numpy(a).cuda()


def to_host_u16(t):
    return t.cpu().numpy().view(np.uint16)


def bf16_to_f64(u16):
    return (np.asarray(u16, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def check_index_sets(idx_gpu, sal_oracle, budget, band=BAND):
    """Per head: the GPU's admitted set must equal the oracle's top-k wherever the
    oracle's k-th and (k+1)-th saliencies differ by more than `band` (relative);
    otherwise every token clearly above the band must be admitted, none clearly below,
    and the set must have exactly k members.  Returns the number of heads that fell in
    the band case."""
    H, N = sal_oracle.shape
    in_band = 0
    for h in range(H):
        got = set(int(x) for x in idx_gpu[h])
        assert len(got) == budget, f"head {h}: {len(got)} distinct indices, expected {budget}"
        assert list(idx_gpu[h]) == sorted(idx_gpu[h]), f"head {h}: indices not ascending"
        if budget == 0 or budget == N:
            assert got == set(range(N)) if budget == N else not got
            continue
        order = sorted(range(N), key=lambda j: (-sal_oracle[h, j], j))
        tau = sal_oracle[h, order[budget - 1]]
        nxt = sal_oracle[h, order[budget]]
        if (tau - nxt) > band * tau:
            assert got == set(order[:budget]), f"head {h}: index set differs from the oracle's"
        else:
            in_band += 1
            hi = {j for j in range(N) if sal_oracle[h, j] > tau * (1 + band)}
            lo = {j for j in range(N) if sal_oracle[h, j] < tau * (1 - band)}
            assert hi <= got, f"head {h}: a clearly salient token is missing"
            assert not (lo & got), f"head {h}: a clearly non-salient token was admitted"
    return in_band
