"""The work-group trace build (libapex_decode_trace.so): the same outputs as
the product library, bit for bit, and a consistent timeline -- every active
work group's prologue, first tiles and end in order, and the units of all
work groups adding up to the call's."""
import ctypes

import numpy as np
import pytest

import apex_workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def test_trace_build_matches_the_product_and_records_a_timeline(torch_cuda):
    torch = torch_cuda
    import paper_2506_03296_amd as A
    from paper_2506_03296_amd import wg_trace
    product = A.load_library()
    trace = wg_trace.load_trace_library()
    case = W.make_host_case([3000, 17, 900, 4500, 0, 1, 2048], 32, 8, seed=31, poison=True)
    dev = "cuda"
    q, k, v = (torch.from_numpy(x).to(dev) for x in (case.q, case.k_cache, case.v_cache))
    bt, lens = torch.from_numpy(case.block_table).to(dev), torch.from_numpy(case.context_lens).to(dev)
    buf = torch.zeros((4096, wg_trace.WORDS), dtype=torch.int64, device=dev)
    outs = {}
    try:
        for name, lib in (("product", product), ("trace", trace)):
            A._LIB = lib
            if name == "trace":
                assert lib.apex_decode_trace_buffer(ctypes.c_void_p(buf.data_ptr()), 4096) == 0
            for workers in (0, 5):
                outs[(name, workers)] = A.decode_attention_ex(q, k, v, bt, lens, case.scale,
                                                              num_workers=workers)
                torch.cuda.synchronize()
                if name == "trace":
                    rows = buf.cpu().numpy()
                    used = rows[:, 3] > 0
                    units = int(sum(-(-int(L) // 16) for L in case.context_lens if L > 0)) * 8
                    assert int(rows[used, 6].sum()) == units
                    act = used & (rows[:, 6] > 0)
                    r = rows[act]
                    assert np.all(r[:, 0] <= r[:, 1]) and np.all(r[:, 1] <= r[:, 2])
                    assert np.all(r[:, 2] <= r[:, 3]) and np.all(r[:, 4] >= 1)
                    if workers == 5:
                        assert act.sum() == 5
                    buf.zero_()
            if name == "trace":
                assert lib.apex_decode_trace_buffer(None, 0) == 0
    finally:
        A._LIB = product
    for workers in (0, 5):
        a, b = outs[("product", workers)], outs[("trace", workers)]
        assert torch.equal(a.view(torch.int16), b.view(torch.int16)), workers
