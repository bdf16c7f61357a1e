"""Group-normalised advantages of the training group (paper Sec. 3.1, Eq. 2)
and the group-mean decomposition of dual-end groups (Sec. 4.1.3, Eq. 3).
TEST INFRASTRUCTURE: the plain statement of what the library's advantage
entry point computes.

A(o_i^j) = (r_i^j - mu(Y_i)) / (sigma(Y_i) + eps) over the k kept
trajectories Y_i of prompt i.

Readings (listed in the design notes): sigma is the population standard
deviation of the group's rewards (the group is the whole set, as for mu);
eps = 1e-6 keeps a group of equal rewards at advantage 0.

Pins (tests/test_oracle_advantage.py): numpy's mean and standard deviation
(library routines), closed forms (advantages sum to 0 and their squares to
k when eps is negligible; equal rewards give 0), invariance under a positive
affine change of the rewards, and the Eq. 3 decomposition of a dual-end
group's mean into its short and long sides.
"""
import math


def group_advantages(rewards, eps=1e-6):
    """rewards: the k rewards of one kept group, in kept order."""
    k = len(rewards)
    mu = math.fsum(float(r) for r in rewards) / k
    var = math.fsum((float(r) - mu) ** 2 for r in rewards) / k
    sd = math.sqrt(var)
    return [(float(r) - mu) / (sd + eps) for r in rewards]


def kept_advantages(kept, reward_of, eps=1e-6):
    """kept: prompt -> list of trajectory ids; reward_of: trajectory id -> reward."""
    return {i: group_advantages([reward_of[g] for g in ids], eps) for i, ids in kept.items()}


def dual_group_mean(r_short, r_long):
    """Eq. 3: mu(Y_dual) = (K mean(r_short) + L mean(r_long)) / (K + L)."""
    K, L = len(r_short), len(r_long)
    ms = math.fsum(r_short) / K if K else 0.0
    ml = math.fsum(r_long) / L if L else 0.0
    return (K * ms + L * ml) / (K + L)
