"""Which residual adds of a chained network run inside a conv's epilogue.

The paper lowers each QNN operator to simpler ones and relies on operator
fusion to run them together (Sec. III-A, III-B).  A qnn.add that closes a
residual block can run inside the kernel of the conv that produces one of
its operands (qnn_plan_set_residual): that conv then stores the sum, its
own output is never written, and the add's separate pass over three
tensors disappears.  This module only decides where that is valid; the
caller sets the residual on the plan and falls back to a separate add
when the plan refuses it."""
from typing import Dict, Sequence, Tuple

Step = Tuple[str, Tuple[str, ...], str]   # (kind, input tensor names, output tensor name)


def residual_fusions(steps: Sequence[Step]) -> Dict[int, Tuple[int, str]]:
    """Pairs residual adds with the convs that can run them.

    `steps` lists the chain in execution order as (kind, inputs, output):
    kind "conv" for a conv or dense whose plan may take a fused add, "add"
    for a two-operand qnn.add, anything else for other steps.  Returns
    {add index: (conv index, residual tensor name)} for every add such that
      * one operand is written by exactly one step, a "conv" before the add,
        and read by no step but the add (the conv's output is then never
        needed on its own);
      * the other operand, the residual, is a chain input or written only
        by steps before that conv (it is complete when the conv runs);
      * the add's output is written by the add alone (the conv may write
        it early).
    When both operands qualify, the conv that runs later takes the add.
    Each conv takes at most one add."""
    writers: Dict[str, list] = {}
    readers: Dict[str, list] = {}
    for i, (_, ins, out) in enumerate(steps):
        writers.setdefault(out, []).append(i)
        for name in ins:
            readers.setdefault(name, []).append(i)
    fused: Dict[int, Tuple[int, str]] = {}
    taken = set()
    for i, (kind, ins, out) in enumerate(steps):
        if kind != "add" or len(ins) != 2 or writers.get(out) != [i]:
            continue
        best = None
        for k in (0, 1):
            op, other = ins[k], ins[1 - k]
            w = writers.get(op, [])
            if len(w) != 1:
                continue
            c = w[0]
            if c >= i or steps[c][0] != "conv" or c in taken or readers.get(op) != [i]:
                continue
            if any(j >= c for j in writers.get(other, [])):
                continue
            if best is None or c > best[0]:
                best = (c, other)
        if best is not None:
            fused[i] = best
            taken.add(best[0])
    return fused
