"""Several host threads driving the library at once, each with its own window, workspace
and stream (include/odb.h allows concurrent calls on distinct streams and workspaces):
every thread's plan, tiles and loss weights equal the oracle's, and each thread's error
message is its own."""
import threading

import numpy as np
import pytest

import oracle
import synth
from _parity import compare_collate_full, compare_loss_weights, compare_plan, log

pytestmark = pytest.mark.gpu


def _window(i):
    rng = np.random.default_rng(300 + i)
    W = 2 + i % 4
    per = [rng.integers(1, 2500, int(rng.integers(1, 4000 if i % 2 else 20000))) for _ in range(W)]
    mode = "nonjoin" if i % 3 == 2 else "join"
    n = sum(len(x) for x in per)
    return synth.window_from_ranks(f"thread_{i}", per, int(rng.choice([4096, 16384, 65536])), mode=mode,
                                   quota=n // 2 if mode == "nonjoin" else 0)


def test_concurrent_host_threads():
    import torch
    import paper_2606_19989_amd as odb

    windows = [_window(i) for i in range(6)]
    refs = [oracle.plan_window(w) for w in windows]
    results, errors = [None] * len(windows), [None] * len(windows)
    start = threading.Barrier(len(windows))
    errs = threading.Barrier(len(windows))

    def work(i):
        try:
            w = windows[i]
            s = torch.cuda.Stream()
            tok_off, toks, ident = synth.device_tensors(w, "cuda")
            win = odb.DeviceWindow(w.rank_off, tok_off, toks, ident, w.num_identities)
            pipe = odb.Pipeline(win, w.budget, mode=w.mode, quota=w.quota, pad_id=i)
            torch.cuda.synchronize()
            start.wait()
            for _ in range(3):   # repeated so the threads' calls interleave
                pipe.form(s)
                pipe.align(s)
                outs = pipe.collate(s)
            s.synchronize()
            odb.odb_collate_status(pipe.ws, s)
            # an argument error on this thread leaves its own message: every thread fails
            # with a different mode before any thread reads its message back
            with pytest.raises(odb.OdbError):
                odb.odb_loss_weights(w.W, 1, 100 + i, pipe.slot_rows, pipe.slot_tokens, None, pipe.slot_tokens, None,
                                     None, s)
            errs.wait()
            msg = odb.load().odb_last_error_message()
            results[i] = (pipe, outs, msg)
        except BaseException as e:   # reported by the main thread
            errors[i] = e

    threads = [threading.Thread(target=work, args=(i,)) for i in range(len(windows))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=300)
    assert not any(t.is_alive() for t in threads), "a thread did not finish"
    for i, e in enumerate(errors):
        if e is not None:
            raise e
    torch.cuda.synchronize()
    for i, (w, ref) in enumerate(zip(windows, refs)):
        pipe, outs, msg = results[i]
        log(f"thread {i}: {w.name} W={w.W} n={w.n} mode={w.mode}")
        compare_plan(w, pipe, ref)
        compare_collate_full(w, outs, ref, i)
        compare_loss_weights(pipe, ref)
        assert msg.decode() == f"unknown loss-weight mode {100 + i}", msg
