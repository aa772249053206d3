"""Brute-force restatement of the Sec. 3.2 mask rules for tiny inputs.

Deliberately written as plain loops over an L x L list-of-lists, rule by rule,
from the paper's text; it shares nothing with ``oracle.mask`` (which is what it
pins).  Segment index sets are recovered here by their own small scan.
"""
NEG = float("-inf")
SYSTEM, TEXT, NEXUS, CURRENT = 0, 1, 2, 3


def segment_sets(role, turn):
    """Return a list of (B_i, N_i) position lists, in sequence order."""
    sets = []
    cur = None
    for p, (r, t) in enumerate(zip(role, turn)):
        if r == TEXT:
            if cur is None or cur[2] != t or cur[1]:
                cur = ([], [], t)
                sets.append(cur)
            cur[0].append(p)
        elif r == NEXUS:
            cur[1].append(p)
        else:
            cur = None
    return [(b, n) for b, n, _ in sets]


def brute_force_mask(role, turn, nexus_scope="all"):
    """nexus_scope "all": Eq.(5) as written; "up_to_own": a Nexus query sees the Nexus
    keys of its own and earlier segments only (reading A3')."""
    L = len(role)
    M = [[NEG] * L for _ in range(L)]
    # Basic causal rule, Eq.(3); applied globally, so mixed text/Nexus pairs too.
    for p in range(L):
        for q in range(L):
            both_nexus = role[p] == NEXUS and role[q] == NEXUS
            if not both_nexus and q <= p:
                M[p][q] = 0.0
    # Historical body removal, Eq.(4).
    for body, nexus in segment_sets(role, turn):
        end = max(nexus) if nexus else max(body)
        for p in range(L):
            if p > end:
                for q in body:
                    M[p][q] = NEG
    # Bidirectional Nexus visibility, Eq.(5).
    seg_of = {}
    for i, (_, nexus) in enumerate(segment_sets(role, turn)):
        for p in nexus:
            seg_of[p] = i
    all_nexus = [p for p in range(L) if role[p] == NEXUS]
    for a in all_nexus:
        for b in all_nexus:
            if nexus_scope == "all" or seg_of[b] <= seg_of[a]:
                M[a][b] = 0.0
    return [[M[p][q] == 0.0 for q in range(L)] for p in range(L)]


def closed_form_row_counts(system, bodies, nexus, current, nexus_scope="all"):
    """Visible keys per query row, derived by hand from the rules for a well-formed layout:
    system row r -> r+1; body row r of segment i -> S + P_i + r + 1 (P_i = Nexus before i);
    Nexus row of segment i -> S + b_i + K_tot (under "up_to_own": S + b_i + P_i + k_i);
    current row r -> S + K_tot + r + 1."""
    counts = [r + 1 for r in range(system)]
    K_tot = sum(nexus)
    P = 0
    for b, k in zip(bodies, nexus):
        counts += [system + P + r + 1 for r in range(b)]
        counts += [system + b + (K_tot if nexus_scope == "all" else P + k)] * k
        P += k
    counts += [system + K_tot + r + 1 for r in range(current)]
    return counts


def read_golden_mask(path):
    roles = turns = None
    rows = []
    with open(path) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            if line.startswith("roles"):
                roles = [int(x) for x in line.split()[1:]]
            elif line.startswith("turns"):
                turns = [int(x) for x in line.split()[1:]]
            else:
                rows.append([x == "1" for x in line.split()])
    return roles, turns, rows
