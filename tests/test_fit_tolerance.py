"""Where the GPU fit's tolerance comes from.

The GPU fit differs from the fp64 oracle mainly by one documented rounding:
each stripped key (source and target) enters the Gram matrices as the sum
of two bf16 numbers, its rounding to bf16 and the rounding of the remainder
(about 16 significant bits; values are used exactly as stored).  This test
refits, in the oracle, on keys stripped in fp64 and then rounded that way,
and checks that the change it causes in W and b stays well inside the GPU
parity tolerance (a tenth of it), on the GPU test's own inputs.  Rounding
the stripped keys to plain bf16 instead would move W by relF 1-2e-2 here."""

import numpy as np
import torch

from oracle import kvx_oracle as O
from paper_2608_03893_amd import synth
from tests.test_gpu_fit import FIT_CASES, TOL_FIT, _relF


def _bf16(x):
    return torch.from_numpy(x).to(torch.bfloat16).double().numpy()


def _hilo(x):
    hi = _bf16(x)
    return hi + _bf16(x - hi)


def test_bf16_rounding_of_stripped_keys_fits_the_tolerance():
    worst = {"K": 0.0, "V": 0.0}
    for name, (cfg, N, *lists) in FIT_CASES.items():
        c = synth.make_calibration(cfg, N, "cpu")
        if lists:
            c["idx"] = np.asarray(lists[0], dtype=np.int32)
        src = c["src"].double().numpy()
        tgt = c["tgt"].double().numpy()
        pos = c["positions"].numpy()
        idx = np.asarray(c["idx"])
        W, b = O.fit_cache(src, idx, tgt, c["rope_src"], c["rope_tgt"], pos, lam=0.01)[0::2]
        # the same fit on stripped keys rounded once to bf16
        Wr = np.zeros_like(W)
        br = np.zeros_like(b)
        for l in range(cfg.L_t):
            for h in range(cfg.H):
                X = np.concatenate([_hilo(O.rope_rotate(src[s, 0, h], pos, c["rope_src"], inverse=True))
                                    for s in idx[l]], axis=1)
                Y = _hilo(O.rope_rotate(tgt[l, 0, h], pos, c["rope_tgt"], inverse=True))
                Wr[l, h], br[l, h] = O.ridge_fit(X, Y, 0.01)
        eW, eb = _relF(Wr, W).max(), _relF(br[:, :, None], b[:, :, None]).max()
        print(f"{name}: rounding moves W_K by relF {eW:.2e}, b_K by {eb:.2e}")
        worst["K"] = max(worst["K"], eW, eb)
    assert worst["K"] <= TOL_FIT["K"] / 10
