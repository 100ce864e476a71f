"""fo_run_overlapped_noalloc on the GPU, through the C ABI: the same outputs
(reordered GEMM output, consumer buffer, restored output) and status as
fo_run_overlapped with a caller-owned counters array, bit for bit, on calls
in a row that share the library's static counters array -- the second with
a smaller input, the third repeating the first."""
import numpy as np
import pytest

import paper_2504_19519_amd as fo
import workloads
from gpu_util import dev_plan, empty16, from_dev, plan_for, say, to_dev, torch_mod, zeros_u32

pytestmark = pytest.mark.gpu

# workload, (M, N, K, modelled CUs, partition in waves)
CASES = [("rs_8192x8192x3584", (1024, 1280, 512, 8, (2, 1))),
         ("a2a_4096x7168x2048", (512, 512, 256, 2, (1, 1))),
         ("rs_8192x8192x3584", (1024, 1280, 512, 8, (2, 1)))]


def _run(w, inp, plan, dp, d, noalloc, s1, s2):
    torch = torch_mod()
    n = w.M * w.N
    C, dst, out = empty16(n, w.dtype), empty16(plan.dest_elems, w.dtype), empty16(n, w.dtype)
    status = zeros_u32(1)
    torch.cuda.synchronize()
    if noalloc:
        fo.run_overlapped_noalloc(plan, dp, d["A"], d["W"], C, d["peer"], dst, out, d["bias"], d["gamma"], w.eps,
                                  w.rmsnorm, status_word=status, gemm_stream=s1, comm_stream=s2)
    else:
        counters = zeros_u32(plan.num_counters)
        fo.run_overlapped(plan, dp, d["A"], d["W"], C, d["peer"], dst, out, d["bias"], d["gamma"], w.eps,
                          w.rmsnorm, counters, status, s1, s2)
    torch.cuda.synchronize()
    return from_dev(C)[:n], from_dev(dst)[:plan.dest_elems], from_dev(out)[:n], int(status.cpu()[0])


def test_noalloc_matches_the_allocating_entry_point():
    torch = torch_mod()
    assert torch.cuda.is_available(), "no GPU visible"
    fo.lib()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for k, (name, (M, N, K, cus, sizes)) in enumerate(CASES):
        w = workloads.WORKLOADS[name].with_shape(M, N, K)
        say(f"[noalloc] call {k}: {w.name} cus={cus} sizes={sizes}")
        inp = workloads.make_inputs(w)
        plan, _ = plan_for(w, inp, num_cus=cus, sizes=list(sizes))
        assert plan.num_counters <= fo.NOALLOC_MAX_COUNTERS
        dp = dev_plan(plan)
        d = {"A": to_dev(inp.A), "W": to_dev(inp.W),
             "peer": to_dev(inp.peer) if w.pattern != "subtoken" else None,
             "bias": to_dev(inp.bias) if inp.bias is not None else None,
             "gamma": to_dev(inp.gamma) if inp.gamma is not None else None}
        ref = _run(w, inp, plan, dp, d, False, s1, s2)
        got = _run(w, inp, plan, dp, d, True, s1, s2)
        assert ref[3] == 0 and got[3] == 0, f"call {k}: status {ref[3]} / {got[3]}"
        for what, a, b in zip(("C'", "dst", "out"), got[:3], ref[:3]):
            np.testing.assert_array_equal(a, b, err_msg=f"call {k}: {what}")
