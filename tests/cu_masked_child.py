"""Child process of tests/test_gpu_cu_masked.py: the stage on CU-masked
streams.  It runs in a fresh process because each masked stream needs a
hardware queue of its own and the runtime gives a process four: the three
masked streams are created first, through the library, and torch creates no
stream here (its work stays on the null stream; events mark the masked
streams through ExternalStream wrappers).

Checks, against the oracle (every row) and bit for bit against the same
micro-batches on the null stream:
  * dispatch, expert FFN and combine of each micro-batch on three streams
    with disjoint CU sets (16, 16 and the rest), chained by events;
  * whole micro-batches submitted on the GEMM stream alone, whose persistent
    grids are sized by its CU count.
"""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))


def log(m):
    print(m, flush=True)


def main():
    import numpy as np
    import torch

    import oracle
    from paper_2606_22541_amd import inputs
    from paper_2606_22541_amd import moe_stage as C
    from paper_2606_22541_amd.stage import ExpertStage, bf16_bits, to_device_routing
    from gpu_common import BF16_TOL, check_outputs

    torch.cuda.set_device(0)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    C.load_library()
    parts = {"dispatch": (0, 16), "combine": (16, 16), "gemm": (32, cus - 32)}
    hs = {}
    for name, (first, n) in parts.items():
        hs[name] = C.moe_stream_create_cu_masked(first, n)
        log("masked stream %s: CUs [%d, %d)" % (name, first, first + n))
    ext = {k: torch.cuda.ExternalStream(v) for k, v in hs.items()}

    cfg = inputs.MoEConfig("cum", d=1024, f=512, E=64, e0=0, E_loc=8, k=8,
                           lengths=(2048, 1500, 777), seed=41)
    w = inputs.make_weights(cfg, "cuda")
    mbs = inputs.make_microbatches(cfg, "cuda")
    ow = oracle.OracleWeights(w, "bf16")
    with ExpertStage(cfg, w, n_slots=4, max_tokens=2048) as st:
        def prep(mb):
            ids, wt = to_device_routing(mb.ids, mb.w)
            out = torch.full((mb.ids.shape[0], cfg.d), float("nan"), dtype=torch.bfloat16,
                             device="cuda")
            return st.microbatch(mb.x, ids, wt, out), (ids, wt, out)

        # reference: whole micro-batches on the null stream
        ref_out = []
        keep = []
        for mb in mbs:
            m, k = prep(mb)
            keep.append(k)
            st.submit(m, 0)
            ref_out.append(k[2])
        st.sync()
        torch.cuda.synchronize()
        # three masked streams: dispatch -> FFN -> combine, chained by events
        tri_out = []
        for i, mb in enumerate(mbs):
            m, k = prep(mb)
            keep.append(k)
            torch.cuda.synchronize()                 # inputs written on the null stream
            st.dispatch(i, m, hs["dispatch"])
            e1 = torch.cuda.Event()
            e1.record(ext["dispatch"])
            ext["gemm"].wait_event(e1)
            st.expert_ffn(i, hs["gemm"])
            e2 = torch.cuda.Event()
            e2.record(ext["gemm"])
            ext["combine"].wait_event(e2)
            st.combine(i, hs["combine"])
            tri_out.append(k[2])
        st.sync()
        torch.cuda.synchronize()
        # whole micro-batches on the GEMM stream alone
        g_out = []
        for mb in mbs:
            m, k = prep(mb)
            keep.append(k)
            torch.cuda.synchronize()
            st.submit(m, hs["gemm"])
            g_out.append(k[2])
        st.sync()
        torch.cuda.synchronize()
        for i, mb in enumerate(mbs):
            ref = oracle.run_stage(cfg, ow, bf16_bits(mb.x), mb.ids, mb.w)
            a, b, c = bf16_bits(ref_out[i]), bf16_bits(tri_out[i]), bf16_bits(g_out[i])
            err = check_outputs(b, ref, BF16_TOL, "masked streams, micro-batch %d" % i)
            assert np.array_equal(a, b), "three masked streams differ from the null stream"
            assert np.array_equal(a, c), "the masked GEMM stream differs from the null stream"
            log("micro-batch %d (T=%d): rel-L2 %.3e, bit-identical on masked streams" % (
                i, mb.ids.shape[0], err))
    for h in hs.values():
        C.moe_stream_destroy(h)
    log("CU-MASKED OK")


if __name__ == "__main__":
    main()
