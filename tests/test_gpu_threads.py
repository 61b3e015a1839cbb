"""Two host threads calling mla_online_attend on their own streams at once: the
plan uploads share the library's per-device staging slots (guarded by a mutex
and an event per slot), so every call must still see its own plan.  Each
thread alternates between two different segment tables; every result must equal
the same call made alone, bit for bit."""
import threading

import numpy as np
import pytest

from workloads import make_custom

pytestmark = pytest.mark.gpu


def _bits(t):
    import torch
    return t.view(torch.int32).clone()


def test_concurrent_attend_calls():
    import torch
    from paper_2609_07008_amd import device_inputs, step
    wls = [make_custom([70, 90, 66], req_perm=[2, 0, 1], tq=12, H=16, G=2, d_c=512, d_r=64, d_model=256,
                       fp32=False, seed=41, prot_frac=0.2),
           make_custom([33, 150], req_perm=[1, 0], tq=7, H=16, G=2, d_c=512, d_r=64, d_model=256,
                       fp32=False, seed=42, prot_frac=0.1)]
    inputs = [device_inputs.upload(wl) for wl in wls]
    # reference: each table alone, on the default stream
    refs = []
    for wl, inp in zip(wls, inputs):
        st = step.OnlineStep(wl.geom, wl.segs, wl.prot_rows, wl.glob_head, 0)
        st.attend(inp["kv"], inp["q_glob"], inp["q_loc"])
        torch.cuda.synchronize()
        refs.append((_bits(st.part_o), _bits(st.part_lse)))

    errors = []

    def worker(tid):
        try:
            s = torch.cuda.Stream()
            steps = [step.OnlineStep(wl.geom, wl.segs, wl.prot_rows, wl.glob_head, 0) for wl in wls]
            for it in range(12):
                k = (it + tid) % 2
                st, inp = steps[k], inputs[k]
                with torch.cuda.stream(s):
                    st.part_o.fill_(float("nan"))
                    st.attend(inp["kv"], inp["q_glob"], inp["q_loc"], stream=s)
                s.synchronize()
                if not (torch.equal(_bits(st.part_o), refs[k][0]) and torch.equal(_bits(st.part_lse), refs[k][1])):
                    errors.append((tid, it, k))
        except Exception as e:   # reported below, in the main thread
            errors.append((tid, repr(e)))

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads)
    assert not errors, errors
