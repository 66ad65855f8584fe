"""The residual-network parity cases (test helper): tests/test_gpu_model6.py
runs them on the GPU, tests/golden/make_resnet_tolerance.py sizes their
tolerance with the oracle alone.  Inputs from the seeded generators of
workload.py."""
from paper_2604_12841_amd import workload

G, R, N = workload.GELU_TANH, workload.RELU, workload.NONE
RESNET_CASES = [
    dict(name="model6_d5", blocks=workload.MODEL6_BLOCKS, d=5, T=5, B=2, layout="paper"),
    dict(name="model6_d3_b1", blocks=workload.MODEL6_BLOCKS, d=3, T=4, B=1, layout="paper"),
    dict(name="w64_paper", blocks=workload.resnet_blocks([64, 64, 64]), d=7, T=5, B=3, layout="paper"),
    dict(name="w64_plaquette_relu", blocks=workload.resnet_blocks([64, 64], c_in=2, act=R), d=5, T=6, B=2,
         layout="plaquette"),
    dict(name="mid_projection", blocks=[(4, 64, 64, G), (64, 128, 128, G), (128, 128, 4, G)], d=5, T=5, B=8,
         layout="paper"),
    dict(name="narrowing", blocks=[(4, 128, 128, G), (128, 64, 64, G), (64, 64, 4, G)], d=5, T=5, B=8,
         layout="paper"),
    dict(name="w256", blocks=workload.resnet_blocks([256, 256]), d=5, T=4, B=2, layout="paper"),
    dict(name="linear_3_blocks", blocks=[(4, 64, 64, N), (64, 64, 64, N), (64, 64, 4, N)], d=5, T=5, B=8,
         layout="paper"),
]


# the cases the fp8 path runs (projections only in the first and the last
# block, where they are fused)
RESNET_FP8_CASES = [c for c in RESNET_CASES if c["name"] not in ("mid_projection", "narrowing")]


def case_inputs(case):
    """(weights, det, first, last) of a case."""
    weights = workload.resnet_weights(case["blocks"], seed=81 + case["d"])
    det, _ = workload.make_inputs(case["d"], case["T"], case["B"], 0.01, 0.01, 82)
    first = last = "Z" if case["layout"] == "paper" else None
    return weights, det, first, last
