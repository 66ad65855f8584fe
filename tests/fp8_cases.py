"""The fp8 parity cases (test helper): the GPU parity tests run them, and
tests/golden/make_fp8_tolerance.py sizes the fp8 tolerance on them with the
oracle alone.  Inputs come from the seeded generators of workload.py."""
from paper_2604_12841_amd import workload

# plaquette cases: benchmark workload id and batch (its weights and
# inputs); paper cases: a model of Table models at d = T (the paper layout,
# Z-basis memory, the benchmark's weight and input seeds)
FP8_CASES = [
    dict(name="w2_b4", layout="plaquette", cfg=2, batch=4),
    dict(name="w2_relu_b2", layout="plaquette", cfg=2, batch=2, act="relu"),
    dict(name="w3_b2", layout="plaquette", cfg=3, batch=2),
    dict(name="m1_d9_b2", layout="paper", model=1, d=9, batch=2),
    dict(name="m4_d7_b2", layout="paper", model=4, d=7, batch=2),
    dict(name="m2_d5_b2", layout="paper", model=2, d=5, batch=2),
    dict(name="m5_d5_b1", layout="paper", model=5, d=5, batch=1),
]


def case_inputs(case):
    """(d, T, layers, weights, det, layout, first, last) of a case."""
    act = workload.RELU if case.get("act") == "relu" else workload.GELU_TANH
    if case["layout"] == "plaquette":
        c = workload.CONFIGS[case["cfg"]]
        layers = workload.config_layers(case["cfg"], act)
        weights = workload.config_weights(case["cfg"], act)
        det, _ = workload.config_inputs(case["cfg"], case["batch"])
        return c["d"], c["T"], layers, weights, det, "plaquette", None, None
    d = T = case["d"]
    layers = workload.paper_model_layers(case["model"], act)
    weights = workload.he_normal_weights(layers, 4000 + case["model"])
    det, _ = workload.make_inputs(d, T, case["batch"], 0.003, 0.003, 5000 + d)
    return d, T, layers, weights, det, "paper", "Z", "Z"
