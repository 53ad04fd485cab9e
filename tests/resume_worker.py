"""One process of the fresh-process resume test (run as a script, not collected).

    python tests/resume_worker.py run  OUT.npz            steps 0..TOTAL-1 in one process
    python tests/resume_worker.py save CKPT.bin           steps 0..SAVE-1, then export the checkpoint
    python tests/resume_worker.py resume CKPT.bin OUT.npz  import, then steps SAVE..TOTAL-1

The stage: two FP8 linears, 8 microbatches of 48 tokens on the zero-bubble
schedule, amax history 4 (several rollovers per step), prebuilt graphs on the
caller's stream.  Between optimizer steps the master weights become
bf16(0.75 W), computed on the host from the initial weights, so every process
can rebuild the weights of any step.  Outputs of the steps from SAVE on (Y,
dX, the placed gradients, the FP8 state) are written to OUT.npz.
"""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

TOTAL, SAVE = 8, 3


def spec():
    from tests.stage_driver import Spec
    return Spec([(96, 160), (72, 200)], tokens=48, M=8, history=4, margin=0, in_dtype="bf16", shared_view=False,
                cfg=2)


def weights_at(sp, step):
    import numpy as np
    import workloads as W
    ws = [sp.weight(u) for u in range(len(sp.shapes))]
    for _ in range(step):
        ws = [W.Tensor(W.f32_to_bf16_bits(w.as_f32() * np.float32(0.75)), "bf16") for w in ws]
    return ws


def main():
    import numpy as np
    import torch
    from paper_2609_23536_amd import qe
    from tests import schedules as S
    from tests.stage_driver import GpuStage

    mode = sys.argv[1]
    sp = spec()
    d = torch.device("cuda:0")
    first = SAVE if mode == "resume" else 0
    last = SAVE if mode == "save" else TOTAL
    g = GpuStage(qe, sp, use_graphs=True, device=d, replay_on_caller=True, weights=weights_at(sp, first))
    assert g.ctx.qe_prebuild_graphs(sp.tokens, qe.BF16, qe.F32, qe.BF16, qe.F32) == "OK"
    if mode == "resume":
        payload = open(sys.argv[2], "rb").read()
        assert g.ctx.qe_checkpoint_import(payload) == "OK"
        st = g.ctx.qe_get_state()
        assert st["e_w"] == SAVE and st["token"] == 0
    out = {}
    for step in range(first, last):
        g.run(S.ZB_STEP0 if step % 2 == 0 else S.ZB_STEP1, step, step)
        torch.cuda.synchronize()
        if step >= SAVE:
            out[f"grad_{step}"] = g.grad.cpu().numpy().copy()
            for (kind, u, m, s), v in g.outs.items():
                out[f"{kind}_{u}_{m}_{s}"] = v.cpu().numpy().copy()
            for u in range(len(sp.shapes)):
                for r, (h, sc, si) in g.fp8_state(u).items():
                    out[f"state_{u}_{r}_{step}"] = np.concatenate([h, np.array([sc, si], dtype=np.float32)])
        g.outs = {}
        g.end_step(weights_at(sp, step + 1))
    assert g.ctx.qe_sync() == "OK"
    st = g.ctx.qe_get_state()
    assert st["device_token"] == st["token"]
    assert st["captures"] == 3 * sp.M * len(sp.shapes)
    if mode == "save":
        cst, payload = g.ctx.qe_checkpoint_export()
        assert cst == "OK"
        with open(sys.argv[2], "wb") as f:
            f.write(payload)
    else:
        np.savez(sys.argv[-1], **out)
    g.ctx.close()
    print(f"resume_worker {mode}: steps {first}..{last - 1} done", flush=True)


if __name__ == "__main__":
    main()
