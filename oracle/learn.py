"""Learning the FSM batching policy (Section 2.3), plain and slow.

TEST INFRASTRUCTURE ONLY (see the package docstring).  Shares no code with the
host library's learner.

The environment is the dataflow graph G of Algorithm 1.  At step t the state
is S_t = E(G_t) (one of the encodings of Section 2.3), the action a_t is a type
present on the frontier, and executing every frontier node of type a_t turns
G_t into G_{t+1}.  An episode runs until every node has executed.

Reward (Eq. 1, with its ratio read the way the worked example of Section 2.3
evaluates it: 5/7 for O and 1/1 for I, a value in (0, 1]):

    r(S_t, a_t) = -1 + alpha * |Frontier_{a_t}(G_t)| / |Frontier(G^{a_t}_t)|

Training is tabular Q-learning with N-step bootstrapping (Section 2.3): the
target of Q(S_tau, a_tau) is the N-step return

    G = sum_{i=tau}^{min(tau+N, T)-1} gamma^(i-tau) r_i
        + [tau + N < T] gamma^N max_a Q(S_{tau+N}, a)

and Q(S_tau, a_tau) += lr * (G - Q(S_tau, a_tau)), updated as soon as
S_{tau+N} is known and, at the end of an episode of T steps, for the
remaining tau in ascending order.  Q starts at 0.  Actions are epsilon-greedy.
Every `check_every` trials (and after the last) the greedy policy
pi(S) = argmax_a Q(S, a) is written out as a table over the visited states and
scheduled; training stops once that schedule reaches the lower bound of
Appendix A.3 (Section 5.4: at most 1000 trials, checked every 50).  The table
returned is the one of the check with the fewest batches (the earliest on
ties).

Choices the paper leaves open (alpha, N, epsilon, the learning rate, gamma,
tie-breaking and the random source) are parameters here with the defaults
below; argmax ties go to the action that comes first in the state key.
Random draws: SplitMix64 (Steele, Lea and Flood, 2014), a counter-based
generator: draw k of seed s is mix(s + (k + 1) * 0x9E3779B97F4A7C15) mod 2^64.
Step c of training (counted over all trials) uses draws 2c (explore when
(draw >> 11) * 2^-53 < epsilon) and 2c + 1 (the explored action is
actions[draw mod len(actions)]).
"""
from __future__ import annotations

from . import schedule as S

_M64 = (1 << 64) - 1
_GAMMA64 = 0x9E3779B97F4A7C15


def splitmix64(seed, k):
    """Output k (k >= 0) of SplitMix64 seeded with `seed` (its published
    definition: a Weyl sequence with increment 0x9E3779B97F4A7C15 passed
    through the variant-13 finalizer of MurmurHash3's 64-bit mix)."""
    z = (seed + (k + 1) * _GAMMA64) & _M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _M64
    return z ^ (z >> 31)


def actions_of(key, encoding):
    """The types a state offers: the frontier types, in key order (E_max's
    trailing majority entry repeats one of them)."""
    return list(key[:-1]) if encoding == S.ENC_MAX else list(key)


def greedy(Q, key, actions):
    """argmax_a Q(S, a); Q defaults to 0; ties to the earliest action."""
    best = actions[0]
    for a in actions[1:]:
        if Q.get((key, a), 0.0) > Q.get((key, best), 0.0):
            best = a
    return best


def greedy_table(Q, encoding):
    """pi(S) for every state S with a Q entry, as {key: type}."""
    keys = sorted({k for (k, _a) in Q})
    return {k: greedy(Q, k, actions_of(k, encoding)) for k in keys}


class _Episode:
    """G_t of Algorithm 1: the executed set and the frontier."""

    def __init__(self, op_type, child_ptr, child_idx, n_types):
        self.op = [int(t) for t in op_type]
        self.ptr, self.idx, self.T = child_ptr, child_idx, n_types
        n = len(self.op)
        self.pending, self.cons = S._consumers(n, child_ptr, child_idx)
        self.pending = [int(p) for p in self.pending]
        self.executed = [False] * n
        self.ready = [set() for _ in range(n_types)]
        for v in range(n):
            if self.pending[v] == 0:
                self.ready[self.op[v]].add(v)
        self.left = n

    def counts(self):
        return [len(r) for r in self.ready]

    def execute(self, a):
        batch = sorted(self.ready[a])
        self.ready[a] = set()
        for v in batch:
            self.executed[v] = True
            for p in self.cons[v]:
                self.pending[p] -= 1
                if self.pending[p] == 0:
                    self.ready[self.op[p]].add(p)
        self.left -= len(batch)


def reward(ep, a, alpha):
    """Eq. 1 for action a in the current G_t."""
    num, den = S.frontier_ratio(ep.op, ep.ptr, ep.idx, ep.executed, a)
    return -1.0 + alpha * (num / den)


def learn(op_type, child_ptr, child_idx, n_types, encoding=S.ENC_SORT, trials=1000,
          check_every=50, n_step=4, alpha=0.5, epsilon=0.1, lr=0.2, gamma=1.0, seed=0):
    """Returns (table, stats, Q): the policy table {key: type}, a dict with
    trials run, the table's batch count, the lower bound and the number of
    states, and the final Q function {(key, type): value}."""
    lb = S.lower_bound(op_type, child_ptr, child_idx, n_types)
    Q = {}
    c = 0                      # training step counter (over all trials)
    best_table, best_nb = {}, None
    trial = 0
    while trial < trials:
        trial += 1
        ep = _Episode(op_type, child_ptr, child_idx, n_types)
        states, acts, rews = [], [], []

        def update(tau, T_end):
            # N-step return from tau (T_end = episode length, or None while running)
            g, mult = 0.0, 1.0
            stop = tau + n_step if T_end is None else min(tau + n_step, T_end)
            for i in range(tau, stop):
                g = g + mult * rews[i]
                mult = mult * gamma
            if T_end is None or tau + n_step < T_end:
                nxt = states[tau + n_step]
                g = g + mult * max(Q.get((nxt, b), 0.0) for b in actions_of(nxt, encoding))
            k = (states[tau], acts[tau])
            q = Q.get(k, 0.0)
            Q[k] = q + lr * (g - q)

        t = 0
        while ep.left > 0:
            key = S.encode_state(ep.counts(), encoding)
            if len(states) == t:
                states.append(key)
            acts_avail = actions_of(key, encoding)
            u = (splitmix64(seed, 2 * c) >> 11) * (1.0 / 9007199254740992.0)
            if u < epsilon:
                a = acts_avail[splitmix64(seed, 2 * c + 1) % len(acts_avail)]
            else:
                a = greedy(Q, key, acts_avail)
            c += 1
            r = reward(ep, a, alpha)
            ep.execute(a)
            acts.append(a)
            rews.append(r)
            t += 1
            if ep.left > 0:
                states.append(S.encode_state(ep.counts(), encoding))
                if t - n_step >= 0:
                    update(t - n_step, None)
            else:
                for tau in range(max(0, t - n_step), t):
                    update(tau, t)
        if trial % check_every == 0 or trial == trials:
            table = greedy_table(Q, encoding)
            batches, _ = S.schedule(op_type, child_ptr, child_idx, n_types, S.POLICY_TABLE,
                                    table=table, encoding=encoding)
            if best_nb is None or len(batches) < best_nb:
                best_table, best_nb = table, len(batches)
            if best_nb <= lb:
                break
    stats = {"trials": trial, "batches": best_nb, "lower_bound": lb, "states": len(best_table)}
    return best_table, stats, Q
