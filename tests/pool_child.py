"""Child process of tests/test_gpu_pool.py: the retrieval side (producer) or
the ranking side (consumer) of a cross-process KV-cache pool.

    python tests/pool_child.py producer|consumer WORKDIR

The producer creates a 3-slot pool, takes slots round-robin, encodes the
users' histories into one slot, synchronises, writes the pool's handle file
and then the slot identifier, and keeps the pool alive until the consumer
reports it is done.  The consumer waits for the slot identifier, maps the
pool from the handle file, ranks every candidate against the slot's cache in
place and saves the scores.  Both build the same seeded inputs.
"""
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

# (hist lens, cand lens, d, H, L, F), seed: shared with the parent test
CASE = ([200, 0, 77, 513], [300, 12, 0, 129], 256, 4, 2, 1024)
SEED = 808
SLOTS, CAPACITY = 3, 1024


def inputs():
    from synth import make_inputs
    hl, kl, d, H, L, F = CASE
    return make_inputs(hl, kl, d, H, L, F, dtype="bf16", seed=SEED, variant="perturbed")


def _wait_for(path, timeout=180.0):
    t0 = time.time()
    while not os.path.exists(path):
        if time.time() - t0 > timeout:
            raise TimeoutError(f"{path} did not appear within {timeout} s")
        time.sleep(0.02)


def _write(path, text):
    with open(path + ".tmp", "w") as f:
        f.write(text)
    os.replace(path + ".tmp", path)


def main():
    role, work = sys.argv[1], sys.argv[2]
    import numpy as np
    import torch
    from paper_2606_00422_amd import upr
    torch.cuda.set_device(0)
    inp = inputs()
    cfg = upr.make_config(inp.d, inp.H, inp.L, inp.F, inp.dtype)
    model = upr.Model(cfg, inp.weights)
    hoff = np.ascontiguousarray(inp.hist_offsets, np.int32)
    coff = np.ascontiguousarray(inp.cand_offsets, np.int32)
    hd, cd = torch.from_numpy(hoff).cuda(), torch.from_numpy(coff).cuda()
    hs, cs = upr.segments(hoff, hd), upr.segments(coff, cd)
    stream = upr.current_stream()
    if role == "producer":
        pool = upr.KvPool.create(cfg, SLOTS, CAPACITY)
        order = [pool.next_slot() for _ in range(4)]
        assert order == [0, 1, 2, 0], order
        slot = pool.next_slot()                              # 1
        X = torch.from_numpy(inp.hist_emb).cuda().to(torch.bfloat16)
        ws = model.workspace(upr.upr_encode_workspace_bytes(model.handle, hs))
        upr.upr_encode_user(model.handle, X.data_ptr(), hs, pool.slot(slot), ws.data_ptr(),
                            ws.numel(), stream)
        torch.cuda.synchronize()
        pool.export_file(os.path.join(work, "pool.handle"))
        _write(os.path.join(work, "slot"), str(slot))
        print(f"producer: encoded into slot {slot}, handle written", flush=True)
        _wait_for(os.path.join(work, "consumer.done"))
        pool.close()
        print("producer: done", flush=True)
    else:
        _wait_for(os.path.join(work, "slot"))
        slot = int(open(os.path.join(work, "slot")).read())
        pool = upr.KvPool.open_file(os.path.join(work, "pool.handle"))
        pcfg, slots, rows = pool.info()
        assert (pcfg.d_model, pcfg.n_layers, slots, rows) == (inp.d, inp.L, SLOTS, CAPACITY)
        C = torch.from_numpy(inp.cand_emb).cuda().to(torch.bfloat16)
        scores = torch.full((int(coff[-1]),), float("nan"), dtype=torch.float32, device="cuda")
        ws = model.workspace(upr.upr_rank_workspace_bytes(model.handle, hs, cs))
        upr.upr_rank_candidates(model.handle, pool.slot(slot), hs, C.data_ptr(), cs,
                                scores.data_ptr(), ws.data_ptr(), ws.numel(), stream)
        torch.cuda.synchronize()
        np.save(os.path.join(work, "scores.npy"), scores.cpu().numpy())
        pool.close()
        _write(os.path.join(work, "consumer.done"), "1")
        print(f"consumer: ranked {int(coff[-1])} candidates from slot {slot}", flush=True)
    model.close()


if __name__ == "__main__":
    main()
