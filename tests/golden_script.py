"""Parser for the hand-worked protocol scripts under tests/golden/."""
import os

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name, with_mode=False):
    """Return (depth, ops, expect) -- and the queue mode (None | ("rr", slots))
    when with_mode. ops: list of (op, learner|None, outcome)."""
    depth, ops, expect, mode = None, [], {}, None
    with open(os.path.join(GOLDEN, name)) as f:
        for raw in f:
            line = raw.split("#", 1)[0].strip()
            if not line:
                continue
            tok = line.split()
            if tok[0] == "depth":
                depth = int(tok[1])
            elif tok[0] == "mode":
                mode = (tok[1], int(tok[2]))
            elif tok[0] == "expect":
                key = tok[1]
                if key == "pulls":
                    expect["pulls"] = int(tok[2])
                    expect["skipped"] = int(tok[4])
                    expect["rejected"] = int(tok[6])
                else:
                    expect[key] = [int(x) for x in tok[2:]]
            else:
                arrow = tok.index("->")
                op = tok[0]
                learner = int(tok[1]) if arrow > 1 else None
                ops.append((op, learner, tok[arrow + 1]))
    if with_mode:
        return depth, ops, expect, mode
    return depth, ops, expect
