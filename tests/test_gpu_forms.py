"""Every launch form of the conv entry points, each on the smallest shape of
a fixed grid that takes it (found with the host-side configuration query):
the output must pass both parity gates against the oracle, a second run
must reproduce it bit for bit, and guard bands around the output buffer
must be left untouched."""
import numpy as np
import pytest

from paper_2003_06513_amd import binding as B
from synthetic import inputs
from gpu_cases import check_output, dev, form_cases, max_terms, note, oracle_ref, prepared_case, torch_mod

pytestmark = pytest.mark.gpu

GUARD = 4096
CANARY = 1234.5


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    B.lib()


CASES = form_cases()


@pytest.mark.parametrize("case", CASES, ids=[str(c[0]).replace(" ", "") + "-" + "x".join(map(str, c[1:6]))
                                             + ("-f16" if c[6] else "-f32") + ("-pool" if c[7] else "")
                                             + "-s%d-a%d" % (c[8], c[9]) for c in CASES])
def test_form_parity_guard_rerun(case):
    torch = torch_mod()
    key, n, cin, cout, h, w, dtc, pool, stride, algo = case
    dtype = np.float16 if dtc == B.PSC_F16 else np.float32
    tdt = torch.float16 if dtc == B.PSC_F16 else torch.float32
    seed = n * 131 + cin * 17 + cout * 5 + h
    wt = inputs.he_weights(seed, cout, cin, dtype)
    masks = B.select_library(wt, 6)
    keep = inputs.keep_after_drop(cout * cin, 50)
    prep, packed = prepared_case(wt, masks, keep)
    got = B.conv3x3_config(prep.layer, dtc, n, h, w, pool, stride, algo)
    if isinstance(key[0], int):
        assert (got["kernel"], got["staged"], got["rows_per_lane"]) == (key[0], key[1], key[5])
    elif key[0] == "stride2":
        assert got["kernel"] == key[1] == 3 and got["cols_per_lane"] == key[2] == (2 if w % 4 == 0 else 1)
    elif key[0] == "wide":
        assert got["kernel"] == key[1] == 1 and got["cols_per_lane"] == key[2] == 4 and got["rows_per_lane"] == 4
    elif key[0] in ("rows", "rows2"):
        assert got["kernel"] == key[1] == 4 and got["cols_per_lane"] == (w - 1) // stride + 1
    else:
        assert got["kernel"] == 2
    x = inputs.normal_activations(seed + 1, (n, cin, h, w), dtype)
    bias = inputs.bias_vector(seed + 2, cout, dtype) if seed % 2 else None
    relu = bool(seed % 3)
    oh, ow = (h // 2, w // 2) if pool else ((h - 1) // stride + 1, (w - 1) // stride + 1)
    numel = n * cout * oh * ow
    buf = torch.full((numel + 2 * GUARD,), CANARY, dtype=tdt, device="cuda")
    y = buf[GUARD:GUARD + numel].view(n, cout, oh, ow)
    xd = dev(x)
    bd = None if bias is None else dev(bias)

    def run():
        if pool:
            B.conv3x3_fwd_pool2(prep.layer, prep.packed, xd, y, bias=bd, relu=relu, algo=algo)
        else:
            B.conv3x3_fwd_strided(prep.layer, prep.packed, xd, y, stride, bias=bd, relu=relu, algo=algo)

    note("form %s shape %s pool=%s stride=%d algo=%d" % (key, (n, cin, cout, h, w), pool, stride, algo))
    run()
    torch.cuda.synchronize()
    first = y.clone()
    y.fill_(-7.0)
    run()
    torch.cuda.synchronize()
    assert torch.equal(first, y), "second run differs"
    assert bool((buf[:GUARD] == CANARY).all()) and bool((buf[GUARD + numel:] == CANARY).all()), \
        "write outside the output"
    ref, s = oracle_ref(x, packed, masks, cout, bias=bias, relu=relu, stride=stride, pool=pool)
    check_output(y.cpu().numpy(), ref, s, dtype, max_terms(packed), "form %s" % (key,))


@pytest.mark.skip(reason="R = 8 rows per lane with several row bands per wave (direct form, fp32, batch 256, "
                         "128@16x16 and 256@8x8) faulted the device once; the cause is not found, so no entry "
                         "point can select it (test_r8_with_several_segments_is_never_planned guards the planner)")
def test_r8_several_segments_direct_form():
    pytest.fail("no entry point selects this form")
