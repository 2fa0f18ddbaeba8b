"""painn_forward_noalloc (the entry point for callers that cannot allocate)
through the C ABI: the same energies as painn_forward, bit for bit, on two
calls in a row with the second on a smaller batch (the fixed scratch keeps
the first call's contents), at every precision; a batch whose workspace
exceeds the fixed scratch and a model not yet packed for the precision are
refused with PAINN_E_ARG."""
import sys

import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _energies(fn, rt, m, g, prec, ds, n):
    out = torch.full((n,), float("nan"), dtype=torch.float64, device=rt.device)
    fn(rt.ctx, m.handle, g.handle, ds.data_ptr() if ds is not None else None, prec,
       out.data_ptr() if n else None)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("name,prec", [("molecules_4096", 1), ("molecules_4096", 2), ("molecules_4096", 0),
                                       ("screening", 2)])
def test_noalloc_matches_forward(name, prec):
    from paper_2604_15380_amd import Runtime
    from paper_2604_15380_amd import binding as B
    say(f"no-alloc forward {name} precision {prec}")
    rt = Runtime(0)
    try:
        hp, W = synth.workload_weights(name)
        m = rt.load_model(synth.weight_file_bytes(hp, W))
        if name == "screening":
            start, _ = synth.screening_batches(3000)[0]
            sizes = [(start, 60), (start + 7, 20)]
        else:
            sizes = [(0, 100), (100, 40)]
        # a model not yet packed for the precision: nothing is packed on this
        # path, so it is refused
        b0 = synth.make_batch(name, *sizes[0])
        inp0 = rt.upload_batch(b0)
        g = rt.build_graph(inp0, hp.cutoff)
        ds0 = inp0["dataset_id"] if hp.n_heads > 1 else None
        with pytest.raises(B.PainnError) as ei:
            _energies(B.painn_forward_noalloc, rt, m, g, prec, ds0, b0.n_struct)
        assert ei.value.status == -1 and "packed" in str(ei.value)
        g.free()
        for start, cnt in sizes:
            b = synth.make_batch(name, start, cnt)
            inp = rt.upload_batch(b)
            g = rt.build_graph(inp, hp.cutoff)
            ds = inp["dataset_id"] if hp.n_heads > 1 else None
            ref = _energies(B.painn_forward, rt, m, g, prec, ds, b.n_struct)
            got = _energies(B.painn_forward_noalloc, rt, m, g, prec, ds, b.n_struct)
            assert np.all(np.isfinite(ref))
            assert np.array_equal(got.view(np.uint64), ref.view(np.uint64)), (start, cnt)
            g.free()
        m.free()
    finally:
        rt.close()


def test_noalloc_refuses_oversized_batch():
    from paper_2604_15380_amd import Runtime
    from paper_2604_15380_amd import binding as B
    say("no-alloc forward, oversized batch")
    rt = Runtime(0)
    try:
        name = "molecules_4096"
        hp, W = synth.workload_weights(name)
        m = rt.load_model(synth.weight_file_bytes(hp, W))
        b = synth.make_batch(name, 0, 1024)        # ~36,000 atoms: beyond 64 MiB at F = 128 FP32
        g = rt.build_graph(rt.upload_batch(b), hp.cutoff)
        ref = _energies(B.painn_forward, rt, m, g, 1, None, b.n_struct)
        with pytest.raises(B.PainnError) as ei:
            _energies(B.painn_forward_noalloc, rt, m, g, 1, None, b.n_struct)
        assert ei.value.status == -1 and "bytes" in str(ei.value)
        # the context and the regular entry point still work
        again = _energies(B.painn_forward, rt, m, g, 1, None, b.n_struct)
        assert np.array_equal(again.view(np.uint64), ref.view(np.uint64))
        # an empty batch needs no workspace
        e = synth.concat([])
        ge = rt.build_graph(rt.upload_batch(e), hp.cutoff)
        B.painn_forward_noalloc(rt.ctx, m.handle, ge.handle, None, 1, None)
        ge.free()
        g.free()
        m.free()
    finally:
        rt.close()
