"""Device copies of a synthetic workload's inputs for the library's calls.

The logits (and, for the fused workload, hidden states and lm_head weight) are filled on the
device by the seeded element generator, the same bits the host generator gives the oracle;
the layout, token ids, K0 offsets and masks are copied from the workload.  Input generation
only: nothing here computes a step of the method.
"""
from __future__ import annotations

import numpy as np

from synth import workloads as W


def device_inputs(wl: W.Workload, with_student: bool = True, device: str = "cuda"):
    import torch
    import paper_2609_14636_amd as P

    stream = torch.cuda.current_stream().cuda_stream
    rto = torch.from_numpy(wl.rollout_turn_off).to(device)
    tto = torch.from_numpy(wl.turn_tok_off).to(device)
    dom = None if wl.domain is None else torch.from_numpy(wl.domain).to(device)
    layout = P.Layout(rto, tto, wl.n_tokens, dom)
    ids = torch.from_numpy(wl.tok).to(device)
    tdt = torch.bfloat16 if wl.dtype == W.BF16 else torch.float32
    N, ld, es = wl.n_tokens, wl.ld, wl.esize
    tboost = torch.from_numpy(wl.teacher_boost).to(device)
    teachers = []
    row_dom = wl.row_domain()
    for d in range(wl.n_teachers):
        t = torch.empty((N, ld), dtype=tdt, device=device)
        rows = np.nonzero(row_dom == d)[0]
        if rows.size:
            splits = np.nonzero(np.diff(rows) != 1)[0] + 1
            for run in np.split(rows, splits):
                a, k = int(run[0]), int(run.size)
                wl.fill_device(t.data_ptr() + a * ld * es, wl.vocab, ld, wl.dtype, a, k,
                               W.teacher_stream(d), wl.teacher_sigma,
                               ids.data_ptr() + 4 * a, tboost.data_ptr() + 4 * a, stream)
        teachers.append(t)
    student = None
    if with_student and wl.student_boost is not None:
        sboost = torch.from_numpy(wl.student_boost).to(device)
        student = torch.empty((N, ld), dtype=tdt, device=device)
        if N:
            wl.fill_device(student.data_ptr(), wl.vocab, ld, wl.dtype, 0, N, W.STREAM_STUDENT,
                           wl.student_sigma, ids.data_ptr(), sboost.data_ptr(), stream)
    mask = None if wl.mask is None else torch.from_numpy(wl.mask).to(device)
    start = None if wl.start is None else torch.from_numpy(wl.start).to(device)
    return dict(layout=layout, ids=ids, teachers=teachers, student=student, mask=mask,
                start=start)


def device_inputs_fused(wl: W.Workload, device: str = "cuda"):
    """Hidden states [N, d], lm_head weight [V, d] and student logits on the device."""
    import torch
    import paper_2609_14636_amd as P

    stream = torch.cuda.current_stream().cuda_stream
    rto = torch.from_numpy(wl.rollout_turn_off).to(device)
    tto = torch.from_numpy(wl.turn_tok_off).to(device)
    layout = P.Layout(rto, tto, wl.n_tokens, None)
    ids = torch.from_numpy(wl.tok).to(device)
    N, d, V = wl.n_tokens, wl.fused_d, wl.vocab
    hidden = torch.empty((N, d), dtype=torch.bfloat16, device=device)
    w = torch.empty((V, d), dtype=torch.bfloat16, device=device)
    if N:
        wl.fill_device(hidden.data_ptr(), d, d, W.BF16, 0, N, W.STREAM_HIDDEN, wl.hidden_sigma,
                       None, None, stream)
    wl.fill_device(w.data_ptr(), d, d, W.BF16, 0, V, W.STREAM_W, wl.w_sigma, None, None, stream)
    sboost = torch.from_numpy(wl.student_boost).to(device)
    student = torch.empty((N, wl.ld), dtype=torch.bfloat16, device=device)
    if N:
        wl.fill_device(student.data_ptr(), V, wl.ld, W.BF16, 0, N, W.STREAM_STUDENT,
                       wl.student_sigma, ids.data_ptr(), sboost.data_ptr(), stream)
    return dict(layout=layout, ids=ids, hidden=hidden, w=w, student=student, mask=None, start=None)
