"""The controller driving the reducer on the GPU, step by step (§4.3
Supervisor recovery, §4.4 route-use budget, §6.4 endpoint guard, §3.2 route
evidence).

Each step the library's Supervisor gives the route policy, nf_route_buckets
reduces every bucket on the GPU, and its decisions and the step's loss go
back to the Supervisor.  Alongside, the oracle controller (oracle/controller.py)
and the oracle reducer run the same loop on the host.  Checked every step:
the two policies, every bucket's decision, the FP32 outputs bit for bit (the
decoded ones as in the other parity tests), and the controllers' states; at
the end the run's route events, alarms, recoveries and modeled traffic."""
import numpy as np
import pytest
import torch

import oracle as nfo
import paper_2606_25759_amd as nf
import synth
from oracle import controller as oc
from tests import nfgpu as H

pytestmark = pytest.mark.gpu

PROFILE = dict(admit_step=3, cooldown_steps=4, guard_steps=3, short_cooldown_steps=0, ema_alpha=0.5,
               slack=1e-3, threshold=2e-2, guard_scale=0.5, near_band=0.0, small_move=0.0,
               target_share=0.9, share_margin=0.02)


@pytest.mark.parametrize("fmt", [nf.NF_FORMAT_BINARY, nf.NF_FORMAT_TERNARY])
def test_controller_drives_route_buckets(fmt):
    W, n, bn = 8, 400_000, 100_032
    lay = synth.small(W, n, 77, bucket_n=bn, elig_frac=0.85, nruns=12)
    g = synth.generate_host(lay)
    m = nfo.mask_from_segments(*synth.mask_segments(lay), n)
    nb = -(-n // bn)
    dev = H.dev()
    gd, md = H.to_dev(g), H.to_dev(m, torch.int64)
    planes = 2 if fmt == nf.NF_FORMAT_TERNARY else 1
    bits = torch.empty((planes * W, (n + 63) // 64), dtype=torch.int64, device=dev)
    counts = torch.empty(planes * n, dtype=torch.uint8, device=dev)
    out = torch.empty(n, dtype=torch.float32, device=dev)
    stats = torch.empty(nb * W * nf.STATS_BYTES, dtype=torch.uint8, device=dev)
    dec = torch.empty(nb * nf.DECISION_BYTES, dtype=torch.uint8, device=dev)
    ws = nf.empty_workspace(nf.nf_workspace_bytes_buckets(W, n, bn), dev)

    # endpoint guard for a full bucket, library against the reference model
    n_e0 = int(H.mask_bool(m, bn).sum())
    model = (2, W // 2, planes, 25e9, 100e9, 20e-6, 30e-6)
    t32, tlow, guard_ok = nf.nf_endpoint_guard(nf.nf_endpoint_model(*model[:3], 0, *model[3:]), bn, n_e0)
    assert (t32, tlow, guard_ok) == oc.endpoint_times(*model, bn, n_e0)

    # a decaying loss with one degradation episode that raises an alarm
    T = 40
    loss = 1.0 - 0.01 * np.arange(T)
    loss[15:21] += np.linspace(0.0, 0.5, 6)
    lp = nf.supervisor_profile(**PROFILE)
    st = nf.nf_supervisor_init(lp)
    sup = oc.Supervisor(PROFILE)
    routes_seen = set()
    for t in range(T):
        pol = nf.nf_supervisor_policy(lp, st, nf.policy(guard_ok=int(guard_ok), format=fmt, tau=0.5))
        adm, veto = sup.policy()
        assert (bool(pol.admitted), bool(pol.veto)) == (adm, veto), f"step {t} policy"
        if t == 25:  # a non-finite gradient appears in bucket 1 from here on
            g[5, bn + 1000] = np.nan
            gd[5, bn + 1000] = float("nan")
        nf.nf_route_buckets(gd, n, bn, md, pol, bits, counts, out, stats, dec, ws)
        d = nf.decisions_host(dec, nb)
        o = out.cpu().numpy()
        opol = H.oracle_policy(pol)
        ref_dec = []
        for b in range(nb):
            a, e = b * bn, min((b + 1) * bn, n)
            gm = np.ascontiguousarray(g[:, a:e])
            mw = np.ascontiguousarray(m[a // 64:(e + 63) // 64])
            ref = (nfo.reduce_bucket_ternary if fmt else nfo.reduce_bucket)(gm, mw, opol)
            rd = ref["decision"]
            H.check_decision(d[b], rd, f"step {t} bucket {b}", exact_scale=bool(fmt))
            routes_seen.add(rd.route)
            mb = H.mask_bool(mw, e - a)
            if rd.route == nfo.ROUTE_L:
                assert H.same_f32(o[a:e][~mb], ref["out"][~mb]), f"step {t} bucket {b} routed values"
                if fmt:
                    assert H.same_f32(o[a:e][mb], ref["out"][mb]), f"step {t} bucket {b} decoded values"
                else:
                    ok, err = H.rel_close(o[a:e][mb], ref["out"][mb])
                    assert ok, f"step {t} bucket {b} decoded values: {err}"
            else:
                assert H.same_f32(o[a:e], ref["out"]), f"step {t} bucket {b} FP32 values"
            ref_dec.append((rd.route, rd.bytes_route, rd.bytes_fp32))
        nf.nf_supervisor_update(lp, st, d, float(loss[t]))
        sup.update(ref_dec, float(loss[t]))
        assert (st.state, st.step, st.cusum, st.smoothed) == (sup.state, sup.step, sup.cusum, sup.smoothed), \
            f"step {t} state"
    assert (st.events_l, st.events_f, st.events_p) == \
        (sup.events[oc.ROUTE_L], sup.events[oc.ROUTE_F], sup.events[oc.ROUTE_P])
    assert (st.alarms, st.readmissions, st.budget_vetoes) == (sup.alarms, sup.readmissions, sup.budget_vetoes)
    assert st.bytes_route == sup.bytes_route and st.bytes_fp32 == sup.bytes_fp32
    # the run went through warm-up (P), the alarm's cooldown and the bad gradient (F), and low-bit (L)
    assert routes_seen == {nfo.ROUTE_L, nfo.ROUTE_F, nfo.ROUTE_P}, routes_seen
    assert st.alarms >= 1 and st.readmissions >= 1
