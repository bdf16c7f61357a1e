"""Token-level streaming, producer side (paper Sec. 4.3.2, App. E).
TEST INFRASTRUCTURE: the plain statement of what the library's chunk
emission computes.

After every sampling step the tokens generated since the last dispatch are
pending; as soon as the pending total reaches the threshold they are
dispatched: one chunk per trajectory that has pending tokens (ascending
trajectory id) holding those tokens (and their log-probabilities), so the
trainer can run its forward pass on a prefix while the suffix is still being
generated.

Readings (listed in the design notes):
* A trajectory that will produce no more tokens (end-of-sequence, truncated
  or aborted) is marked final in the first dispatch after it ended; its chunk
  may then hold zero tokens.  The trainer learns which ones were kept from
  the selection's kept sets.
* Every generated token is streamed, aborted trajectories' included (their
  final mark tells the trainer to drop them).
* When every prompt's kept set is complete, whatever is pending is flushed
  regardless of the threshold.

Pins (tests/test_oracle_streaming.py): per trajectory the concatenation of
its chunks equals its full token history (nothing lost, nothing repeated),
dispatches happen exactly at the steps where the pending total first reaches
the threshold, every trajectory is marked final exactly once, and a threshold
of 1 reproduces sample-level-per-step delivery.
"""


def stream_chunks(length, tokens, logprobs, status, n_steps, threshold):
    """Simulate the dispatches of a finished rollout.

    length: traj -> generated count (trajectory g emits its token t at
    sampling step t + 1 and is final after step length[g]); tokens /
    logprobs: traj -> per-token lists; status: traj -> final status.
    Returns a list of (step, [(traj, start, tokens, logprobs, final_status or 0)]).
    """
    sent = {g: 0 for g in length}
    fin_sent = {g: False for g in length}
    out = []
    for s in range(1, n_steps + 1):
        pending = sum(min(length[g], s) - sent[g] for g in length)
        flush = s == n_steps
        if pending < threshold and not (flush and (pending > 0 or not all(fin_sent.values()))):
            continue
        chunks = []
        for g in sorted(length):
            upto = min(length[g], s)
            final = length[g] <= s
            if upto > sent[g] or (final and not fin_sent[g]):
                chunks.append((g, sent[g], list(tokens[g][sent[g]:upto]),
                               list(logprobs[g][sent[g]:upto]), status[g] if final else 0))
                sent[g] = upto
                if final:
                    fin_sent[g] = True
        out.append((s, chunks))
    return out
