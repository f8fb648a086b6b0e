"""Readers for the hand-derived fixtures under tests/golden/."""
import os

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def read_trace(name):
    """Yields (op, args list, expected string) for each non-comment line."""
    out = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            parts = line.split()
            op = parts[0]
            # args run until the first token that starts an expectation
            i = 1
            args = []
            while i < len(parts) and parts[i] not in ("admit", "refuse", "act", "model", "empty", "-"):
                args.append(int(parts[i]))
                i += 1
            if i < len(parts) and parts[i] == "-" and op in ("get", "release") and not args:
                i += 1  # the args placeholder
            expected = " ".join(parts[i:]) if i < len(parts) else "-"
            out.append((op, args, expected))
    return out


def read_weights():
    rows = []
    with open(os.path.join(GOLDEN, "agg_weights_c1.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                a, s, w = line.split()
                rows.append((float(a), int(s), float(w)))
    return rows


def fmt_get(r, K, with_slot):
    """Formats a scheduler get() result like the fixtures do."""
    if r is None:
        return "empty"
    if r[0] == "model":
        return f"model k={r[1]} tk={r[2]}"
    _, k, seq, slot, c = r
    s = f"act k={k} seq={seq}"
    if with_slot:
        s += f" slot={slot}"
    return s + " c=" + ",".join(str(x) for x in c)
