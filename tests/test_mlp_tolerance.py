"""Where the GPU MLP mapper's tolerance comes from.

The GPU evaluates each network in bf16 with fp32 accumulation.  Four values
are rounded once to bf16 (round-to-nearest-even) on the key path (stripped
input, both hidden activations, output) and three on the value path.  This
test replays exactly those roundings in fp64 on the parity cases' inputs,
one network at a time, and compares the result with the unrounded oracle.
The change must stay within two thirds of the GPU tolerance, leaving the rest
for fp32 accumulation and fp32 RoPE coefficients.  It must also be of the size
the rounding count predicts: above one rounding's effect and below twice the
four-rounding estimate."""

from paper_2608_03893_amd import synth
from tests.test_gpu_mlp import MLP_CASES, TOL_MLP, bf16_replay_layer, oracle_layer, rel_errors


def test_bf16_evaluation_fits_the_tolerance():
    worst_k = worst_v = 0.0
    for name, (cfg, F) in MLP_CASES.items():
        inp = synth.make_mlp_inputs(cfg, F, "cpu")
        for l in range(cfg.L_t):
            err = rel_errors(bf16_replay_layer(inp, l), oracle_layer(inp, l))
            worst_k = max(worst_k, float(err[0].max()))
            worst_v = max(worst_v, float(err[1].max()))
        print(f"{name}: bf16 evaluation relF K {worst_k:.2e}, V {worst_v:.2e}")
    assert worst_k <= TOL_MLP * 2 / 3 and worst_v <= TOL_MLP * 2 / 3
    # one bf16 rounding alone moves a tensor by about 1.6e-3; four by about 3.2e-3
    assert 1.0e-3 < worst_v < 2 * 3.2e-3 and 1.0e-3 < worst_k < 2 * 3.2e-3
