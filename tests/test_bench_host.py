"""Host-side pieces of bench.py that need no GPU: the dense bf16 weight the
bf16 GEMM comparator reads, bf16(dequant(W_Q) + W_O) (eq. 1 and eq. 3),
checked bit for bit against the oracle's dequantisation on the same
synthetic problem."""

import numpy as np
import torch

import bench
import oracle
from synth import make_problem


def test_comparator_weight_matches_oracle():
    K, N = 512, 192
    p = make_problem(1, K, N, frac=0.02, seed=11)
    Wq = torch.from_numpy(p.Wq.view(np.int32).copy())
    s = torch.from_numpy(p.scales.view(np.int16).copy()).view(torch.float16)
    z = torch.from_numpy(p.zeros.view(np.int32).copy())
    w = bench.bf16_dequant_weight(torch, Wq, s, z, p.k, p.n, p.v, K, N)
    assert w.dtype == torch.bfloat16 and tuple(w.shape) == (K, N)
    ref = oracle.dequant(p.Wq, p.scales, p.zeros, K, N, 128)
    np.add.at(ref, (p.k, p.n), oracle.bf16_to_f64(p.v))
    want = oracle.bf16_rne_bits(ref)
    got = w.view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, want)
    # an outlier position holds exactly the outlier (its code is the zero-point)
    assert np.array_equal(got[p.k, p.n], p.v)
