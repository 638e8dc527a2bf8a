"""The layer table against numbers the paper prints (tests/golden/paper_values.json)."""
from paper_2609_10632_amd import workloads as W


def test_parameter_count_and_tensors(golden):
    params = tensors = 0
    for l in W.backbone_neck_layers():
        params += l.params() + 2 * l.co  # conv weight, BN gamma and beta
        tensors += 3
    for l, has_bn, has_bias in W.faithful_head_param_tensors():
        params += l.params() + (2 * l.co if has_bn else 0) + (l.co if has_bias else 0)
        tensors += 1 + (2 if has_bn else 0) + (1 if has_bias else 0)
    assert round(params / 1e6, 1) == golden["parameters_millions"]["value"]
    assert tensors == golden["parameter_tensors"]["value"]


def test_head_locations_and_strides(golden):
    size = golden["input_size"]["value"]
    spatial = [h for h, _ in W.HEAD_SCALES]
    assert [size // h for h in spatial] == golden["strides"]["value"]
    assert sum(h * h for h in spatial) == golden["candidate_locations"]["value"]


def test_layer_chain_is_consistent():
    L = {l.name: l for l in W.backbone_neck_layers()}
    assert len(L) == 65
    # every stride-2 conv halves the spatial size; C2f inner convs keep half the width
    for l in L.values():
        assert l.ho == (l.h // l.s)
    assert L["b1"].h == L["b0"].ho and L["b2.cv1"].h == L["b1"].ho
    assert L["n12.cv1"].ci == L["b9.cv2"].co + L["b6.cv2"].co
    assert L["n21.cv1"].ci == L["n19"].co + L["b9.cv2"].co


def test_flop_totals(golden):
    w4 = W.workload(4)
    assert w4.n == golden["per_gpu_batch"]["value"]
    assert abs(w4.gemm_flops() / 1e9 - 3017.30) < 0.01
    assert abs(W.workload(5).gemm_flops() / 1e9 - 6702.94) < 0.01

