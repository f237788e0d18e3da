"""Independent derivations of the index traces, used to pin the oracle and the GPU path.

Each function takes ops [T] (one element) and returns the traces as Python lists.
"""


def list_stack(ops):
    """A literal list of producer steps: push appends, pop removes, hold does nothing."""
    st = [-1]
    top, ptr = [], [0]
    for t, op in enumerate(ops):
        if op == 1:
            st.append(t)
        elif op == -1:
            if len(st) == 1:
                raise ValueError("underflow")
            st.pop()
        top.append(st[-1])
        ptr.append(len(st) - 1)
    return top, ptr


def alg1_int_stack(ops):
    """Algorithm 1 on an int stack: write t at slot p+1 every step, move p by op, read slot p."""
    S = [-1] + [None] * len(ops)
    p = 0
    top, ptr = [], [0]
    for t, op in enumerate(ops):
        S[p + 1] = t
        p += op
        if p < 0:
            raise ValueError("underflow")
        top.append(S[p])
        ptr.append(p)
    return top, ptr


def parent_pointer(ops):
    """Recurrence on producers: push -> t; hold -> src[t]; pop -> src[src[t]]; src[t+1] = top[t]."""
    src = [-1]
    top = []
    for t, op in enumerate(ops):
        s = src[t]
        if op == 1:
            tp = t
        elif op == 0:
            tp = s
        else:
            if s < 0:
                raise ValueError("underflow")
            tp = src[s]
        top.append(tp)
        src.append(tp)
    return top, src[:-1]


def closed_form(ops):
    """top[t] = latest t' <= t with op[t'] = push and ptr[t'+1] = ptr[t+1]; -1 when ptr[t+1] = 0."""
    ptr = [0]
    for op in ops:
        ptr.append(ptr[-1] + op)
    top = []
    for t in range(len(ops)):
        d = ptr[t + 1]
        if d == 0:
            top.append(-1)
            continue
        tp = -1
        for u in range(t, -1, -1):
            if ops[u] == 1 and ptr[u + 1] == d:
                tp = u
                break
        top.append(tp)
    return top, ptr
