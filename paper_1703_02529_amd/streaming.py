"""Chunked, double-buffered run of one video through the cascade on two HIP streams.

Frames arrive in chunks (from a decoder, a camera or a generator).  Two frame
buffers alternate: while the cascade stream runs chunk k out of one buffer, the
fill stream writes chunk k+1 into the other.  Events order the two streams: the
cascade on a buffer waits for that buffer's fill, and the next fill of a buffer
waits for the cascade that read it.  Between chunks the carried state (area
sums and decisions of the last delta frames) continues the reuse of frame
t - delta across the boundary (Sec. 5), so the chunked result equals a one-shot
run of the whole video.  Frames are batched for the GPU (Sec. 7); larger
chunks raise throughput and add latency on live video (Sec. 8).

With batch_chunks = m > 1 the chunks are staged: each chunk's area sums go
into a batch of m chunks (after which its frame buffer is free for the next
fill), and the detector, compaction, CNN and label resolution run once per
batch, so the CNN sees the survivors of m chunks together.  A chunk's labels
then exist only once its batch is finished.

Streams are created at the default priority.  Nothing here computes: filling
is the caller's `produce` callback, and every cascade step runs in libnsc.
"""
from __future__ import annotations

from typing import Callable, Optional

import torch

from . import nsc_cascade_finish, nsc_cascade_run, nsc_cascade_stage
from .runner import CascadeRunner

# produce(buf, t0, m, stream): enqueue on `stream` the writing of frames
# [t0, t0 + m) into buf (contiguous uint8, frame after frame)
Producer = Callable[[torch.Tensor, int, int, torch.cuda.Stream], None]


class StreamingCascade:
    def __init__(self, wl, blob, chunk: int, lr_w: Optional[torch.Tensor] = None,
                 ref_sums: Optional[torch.Tensor] = None, device="cuda", batch_chunks: int = 1,
                 cnn_pass: int = 0):
        if chunk <= 0 or batch_chunks <= 0:
            raise ValueError("chunk and batch_chunks must be positive")
        self.wl = wl
        self.chunk = chunk
        self.batch_chunks = batch_chunks
        self.device = torch.device(device)
        self.frame_bytes = wl.video.h * wl.video.w * 3
        batch = batch_chunks > 1
        self.runner = CascadeRunner(wl, blob, max_frames=chunk * batch_chunks, lr_w=lr_w,
                                    ref_sums=ref_sums, device=self.device, batch=batch,
                                    cnn_pass=cnn_pass)
        self.bufs = [torch.empty(chunk * self.frame_bytes, dtype=torch.uint8, device=self.device)
                     for _ in range(2)]
        self.s_fill = torch.cuda.Stream(self.device)
        self.s_run = torch.cuda.Stream(self.device)

    def run(self, n_total: int, produce: Producer, label: torch.Tensor, defer: torch.Tensor,
            score: Optional[torch.Tensor] = None, fire: Optional[torch.Tensor] = None,
            logit: Optional[torch.Tensor] = None, timing: bool = False, t_start: int = 0,
            overlap: bool = True, stage_events: Optional[Callable[[int], list]] = None):
        """Runs frames [t_start, t_start + n_total) in chunks; per-frame outputs
        (device tensors of at least n_total entries, indexed from t_start) are
        written in place.  t_start is 0 or the frame where the previous run
        ended (the carried state continues from there).

        overlap=False fills a buffer only after the previous chunk's cascade has
        finished, so that each chunk's cascade runs alone on the GPU.  Returns,
        when `timing` is set, cascade_ms (sum over chunks of the cascade
        stream's time per chunk, the waits for fills excluded; with overlap it
        includes slowdown from sharing the GPU with the fills) and wall_ms
        (first fill to last result).  stage_events(k), when given, returns the
        NSC_STAGE_EVENTS raw event handles that chunk k's cascade (with
        batches: batch k's finishing call) records at its stage boundaries;
        with batches the timing also gives stage_ms, the summed time of the
        chunks' area stages."""
        for name, t in (("label", label), ("defer", defer), ("score", score), ("fire", fire),
                        ("logit", logit)):
            if t is not None and t.numel() < n_total:
                raise ValueError(f"{name} holds {t.numel()} entries, fewer than {n_total} frames")
        filled = [torch.cuda.Event() for _ in range(2)]
        consumed = [torch.cuda.Event() for _ in range(2)]
        starts, ends = [], []
        wall0 = wall1 = None
        if timing:
            wall0 = torch.cuda.Event(enable_timing=True)
            wall1 = torch.cuda.Event(enable_timing=True)
        # the caller's earlier work (allocation, zeroing of outputs) comes first
        cur = torch.cuda.current_stream(self.device)
        self.s_fill.wait_stream(cur)
        self.s_run.wait_stream(cur)
        if timing:
            wall0.record(self.s_fill)
        r = self.runner
        batched = self.batch_chunks > 1
        stage_marks = []   # (start, end) events of the batched area stages
        u_batch = 0        # first frame (relative to t_start) of the open batch

        def outs(sl):
            return dict(score=score[sl] if score is not None else None,
                        fire=fire[sl] if fire is not None else None,
                        logit=logit[sl] if logit is not None else None)

        def timed(fn):
            if timing:
                starts.append(torch.cuda.Event(enable_timing=True))
                ends.append(torch.cuda.Event(enable_timing=True))
                starts[-1].record(self.s_run)
            fn()
            if timing:
                ends[-1].record(self.s_run)

        n_chunks = -(-n_total // self.chunk)
        for k, u0 in enumerate(range(0, n_total, self.chunk)):
            b = k & 1
            m = min(self.chunk, n_total - u0)
            t0 = t_start + u0
            if overlap and k >= 2:
                self.s_fill.wait_event(consumed[b])
            elif not overlap and k >= 1:
                self.s_fill.wait_event(consumed[b ^ 1])
            produce(self.bufs[b], t0, m, self.s_fill)
            filled[b].record(self.s_fill)
            self.s_run.wait_event(filled[b])
            if not batched:
                sl = slice(u0, u0 + m)
                timed(lambda: nsc_cascade_run(
                    r.cfg, r.cnn, self.bufs[b], m, t0, r.state, r.ws, label[sl], defer[sl],
                    stage_events=stage_events(k) if stage_events is not None else None,
                    stream=self.s_run, **outs(sl)))
                consumed[b].record(self.s_run)
                continue
            timed(lambda: nsc_cascade_stage(r.cfg, r.cnn, r.max_frames, r.cnn_pass, self.bufs[b], m,
                                            u0 - u_batch, r.ws, stream=self.s_run))
            if timing:
                stage_marks.append((starts[-1], ends[-1]))
            consumed[b].record(self.s_run)
            if (k + 1) % self.batch_chunks == 0 or k + 1 == n_chunks:
                nb = u0 + m - u_batch
                sl = slice(u_batch, u_batch + nb)
                j = k // self.batch_chunks
                timed(lambda: nsc_cascade_finish(
                    r.cfg, r.cnn, r.max_frames, r.cnn_pass, nb, t_start + u_batch, r.state, r.ws,
                    label[sl], defer[sl],
                    stage_events=stage_events(j) if stage_events is not None else None,
                    stream=self.s_run, **outs(sl)))
                # the buffer's next fill also waits for the batch's finish (so
                # that without overlap the finish, too, runs alone)
                consumed[b].record(self.s_run)
                u_batch += nb
        if timing:
            wall1.record(self.s_run)
        cur.wait_stream(self.s_run)
        cur.wait_stream(self.s_fill)
        if not timing:
            return None
        wall1.synchronize()
        res = dict(chunks=n_chunks,
                   cascade_ms=sum(s.elapsed_time(e) for s, e in zip(starts, ends)),
                   wall_ms=wall0.elapsed_time(wall1))
        if batched:
            res["batches"] = -(-n_chunks // self.batch_chunks)
            res["stage_ms"] = sum(s.elapsed_time(e) for s, e in stage_marks)
        return res

    def close(self):
        self.runner.close()


__all__ = ["StreamingCascade"]
