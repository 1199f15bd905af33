"""Head/group bookkeeping of the key compression (Sec. III-C).

The key projection W^(k) (m x n, n = h * d_h) is split column-wise into K
groups of whole heads; group i holds h_i heads, the h_i sum to h, and the head
ratio is alpha_i = h_i / h.  Group i is factored as L_i (m x r_i) times
R_i (r_i x h_i d_h).  The value projection is factored whole (Sec. III-D).

Readings where the paper is silent:
  * the heads of a group are ordered by ascending head index, so the j-th
    head of group g owns columns [j d_h, (j+1) d_h) of R_g;
  * the grouped heads are the key/value heads; a query head h reads KV head
    floor(h / (H_q / H_kv)) (grouped-query attention, contiguous blocks);
  * group g's latent occupies columns [koff_g, koff_g + r_g) of the per-token
    key latent, with koff_g the sum of the ranks of the groups before g.
"""

from __future__ import annotations

from dataclasses import dataclass
from fractions import Fraction
from typing import List, Sequence


class PartitionError(ValueError):
    pass


def group_members(group_of_kv: Sequence[int], num_groups: int) -> List[List[int]]:
    """Heads of each group, ascending.  Raises unless the groups partition the
    heads: every head in exactly one group and no group empty (Sec. III-C:
    the group sizes sum to h)."""
    members: List[List[int]] = [[] for _ in range(num_groups)]
    for kv, g in enumerate(group_of_kv):
        if not (0 <= int(g) < num_groups):
            raise PartitionError(f"head {kv} assigned to group {g} outside [0,{num_groups})")
        members[int(g)].append(kv)
    for g, mem in enumerate(members):
        if not mem:
            raise PartitionError(f"group {g} has no heads")
    if sum(len(mem) for mem in members) != len(group_of_kv):
        raise PartitionError("group sizes do not sum to the head count")
    return members


@dataclass
class Book:
    hidden: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    ranks: List[int]
    value_rank: int
    members: List[List[int]]
    heads_per_group: List[int]
    alpha: List[Fraction]
    group_of_kv: List[int]
    pos_in_group: List[int]
    koff: List[int]          # [G]   latent column offset of group g
    roff: List[int]          # [G+1] element offset of R_g in the concatenated R blocks
    q_per_kv: int
    kv_of_q: List[int]       # [H_q]
    group_of_q: List[int]    # [H_q]
    qoff: List[int]          # [H_q+1] offset of head h's folded query (r_{g(h)} wide)

    @property
    def num_groups(self) -> int:
        return len(self.ranks)

    @property
    def key_rank_total(self) -> int:
        return sum(self.ranks)

    @property
    def kv_dim(self) -> int:
        return self.num_kv_heads * self.head_dim


def make_book(hidden: int, num_q_heads: int, num_kv_heads: int, head_dim: int,
              group_of_kv: Sequence[int], ranks: Sequence[int], value_rank: int) -> Book:
    G = len(ranks)
    if len(group_of_kv) != num_kv_heads:
        raise PartitionError("group map length differs from the KV head count")
    if num_kv_heads <= 0 or num_q_heads % num_kv_heads != 0:
        raise PartitionError("query heads must be a multiple of KV heads")
    members = group_members(group_of_kv, G)
    sizes = [len(mem) for mem in members]
    for g, (r, hg) in enumerate(zip(ranks, sizes)):
        # a rank-r factorisation of an m x h_g d_h block needs r <= min(m, h_g d_h)
        if not (1 <= r <= min(hidden, hg * head_dim)):
            raise PartitionError(f"rank {r} of group {g} outside [1, min(m, h_g d_h)]")
    if not (1 <= value_rank <= min(hidden, num_kv_heads * head_dim)):
        raise PartitionError("value rank outside [1, min(m, n)]")
    pos = [0] * num_kv_heads
    for mem in members:
        for j, kv in enumerate(mem):
            pos[kv] = j
    koff, acc = [], 0
    for r in ranks:
        koff.append(acc)
        acc += r
    roff, acc = [0], 0
    for r, hg in zip(ranks, sizes):
        acc += r * hg * head_dim
        roff.append(acc)
    qpk = num_q_heads // num_kv_heads
    kv_of_q = [h // qpk for h in range(num_q_heads)]
    group_of_q = [int(group_of_kv[kv]) for kv in kv_of_q]
    qoff, acc = [0], 0
    for h in range(num_q_heads):
        acc += ranks[group_of_q[h]]
        qoff.append(acc)
    return Book(hidden=hidden, num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
                head_dim=head_dim, ranks=list(ranks), value_rank=value_rank, members=members,
                heads_per_group=sizes, alpha=[Fraction(s, num_kv_heads) for s in sizes],
                group_of_kv=[int(g) for g in group_of_kv], pos_in_group=pos, koff=koff,
                roff=roff, q_per_kv=qpk, kv_of_q=kv_of_q, group_of_q=group_of_q, qoff=qoff)


def book_for(wl) -> Book:
    """Book of a workload description (any object with the Workload fields)."""
    return make_book(wl.hidden, wl.num_q_heads, wl.num_kv_heads, wl.head_dim,
                     wl.group_of_kv, wl.group_rank, wl.value_rank)
