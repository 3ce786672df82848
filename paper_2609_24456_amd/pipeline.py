"""Off-policy iteration loop with the experience path scheduled on its own
stream (paper Sec. 4 decoupling of ingestion and delivery; Sec. 6 timing and
granularity).

One compute stream runs the actor's rollout and the learner's update; one
experience stream runs every experience operator -- ingestion, delivery
(sample + gather with importance weights) and priority updates -- in a fixed
program order, so the data they produce does not depend on timing: only *when*
they run changes with the mode (Sec. 4.3: scheduling changes when and where
experience handling runs, not what it produces).

A mode is (overlap_ing, g_ing, overlap_del, g_del):
  g_ing        rollout units ingested per ingestion invocation (an invocation
               runs once g_ing units have accumulated, and at the end);
  overlap_ing  0: the actor waits for each ingestion before its next rollout;
               1: ingestion runs while the actor continues;
  g_del        training batches prepared per delivery invocation: one
               stratified sample of g_del * B transitions (one IS-weight
               normalisation), split into g_del batches in order;
  overlap_del  0: a delivery starts after the rollout of the iteration that
               needs it and the learner waits for it, and the next rollout
               waits for the learner's priority update; 1: the next delivery
               is issued ahead, so it runs during the learner's update.
Off-policy only (integer granularities): replay semantics allow the staleness
batching and prefetching introduce (Sec. 4.1-4.2).

This module only orders calls and events; every experience operation is a call
into the C library through the callables the caller passes in.
"""
from dataclasses import dataclass

import torch


@dataclass(frozen=True)
class Mode:
    overlap_ing: int
    g_ing: int
    overlap_del: int
    g_del: int


def run(mode, iters, rollout, learn, ingest, deliver, update_prio):
    """Run `iters` iterations.

    rollout(t), learn(t): enqueue the actor's / learner's compute for iteration
    t on the current stream (the compute stream).
    ingest(first, n, stream), deliver(k, first, n, stream), update_prio(t, stream):
    enqueue the experience operators on `stream` (a hipStream_t handle):
    ingest rollout units [first, first + n); deliver group k, the batches of
    iterations [first, first + n); apply the learner's priorities of iteration t.
    Returns (elapsed milliseconds, op log in experience-stream order).
    """
    if mode.g_ing < 1 or mode.g_del < 1:
        raise ValueError("off-policy granularities are integers >= 1")
    comp = torch.cuda.Stream()
    exp = torch.cuda.Stream()
    h_exp = exp.cuda_stream
    log = []
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)

    def mark(stream):
        e = torch.cuda.Event()
        e.record(stream)
        return e

    torch.cuda.synchronize()
    start.record(comp)
    exp.wait_event(mark(comp))
    delivered = {}
    first_pending = 0

    def issue_delivery(k):
        first = k * mode.g_del
        n = min(iters, first + mode.g_del) - first
        deliver(k, first, n, h_exp)
        log.append(("deliver", k, first, n))
        delivered[k] = mark(exp)

    for t in range(iters):
        with torch.cuda.stream(comp):
            rollout(t)
        ev_roll = mark(comp)
        # ingestion of the accumulated rollout units
        if t + 1 - first_pending == mode.g_ing or t == iters - 1:
            exp.wait_event(ev_roll)
            ingest(first_pending, t + 1 - first_pending, h_exp)
            log.append(("ingest", first_pending, t + 1 - first_pending))
            ev_ing = mark(exp)
            first_pending = t + 1
            if not mode.overlap_ing:
                comp.wait_event(ev_ing)
        # delivery of the batch the learner needs now
        k = t // mode.g_del
        if k not in delivered:
            if not mode.overlap_del:
                exp.wait_event(ev_roll)
            issue_delivery(k)
        comp.wait_event(delivered[k])
        with torch.cuda.stream(comp):
            learn(t)
        ev_learn = mark(comp)
        # prefetch the next group during the update
        if mode.overlap_del and (t + 1) % mode.g_del == 0 and t + 1 < iters:
            issue_delivery((t + 1) // mode.g_del)
        # the learner's new priorities
        exp.wait_event(ev_learn)
        update_prio(t, h_exp)
        log.append(("prio", t))
        ev_prio = mark(exp)
        if not mode.overlap_del:
            comp.wait_event(ev_prio)
    comp.wait_event(mark(exp))
    end.record(comp)
    torch.cuda.synchronize()
    return start.elapsed_time(end), log
