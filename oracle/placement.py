"""Reference oracle for experience-buffer placement -- TEST INFRASTRUCTURE ONLY.

Plain Python (fp64) statement of Sec. 5 of the paper:

* Sec. 5.1 (Transfer-Latency Model): a placement p costs each sample two
  transfers, actor -> p (ingestion) and p -> learner GPU (delivery), each the
  per-sample size x over the effective bandwidth of that leg.
* Sec. 5.2, Eq. (placement_opt_clean): the placement of least transfer latency
  among those whose memory holds C_buf * x.
* Alg. 1: a linear scan over the candidates keeping the feasible one of least
  latency; a later candidate replaces the kept one only if strictly faster.

Only ``tests/`` may import this module.  It shares no code with the library.
"""
import math


def transfer(x, bw_in, bw_out):
    """Sec. 5.1: per-sample transfer latency of one placement (seconds)."""
    return x / bw_in + x / bw_out


def scan(candidates, capacity, x, bw_in, bw_out, mem):
    """Alg. 1 over ``candidates`` (keys into the per-placement tables
    ``bw_in``, ``bw_out`` and ``mem``): (chosen key or None, latency of each
    candidate)."""
    best, t_min = None, math.inf
    latencies = []
    for p in candidates:
        t = transfer(x, bw_in[p], bw_out[p])
        latencies.append(t)
        if capacity * x <= mem[p] and t < t_min:
            best, t_min = p, t
    return best, latencies
