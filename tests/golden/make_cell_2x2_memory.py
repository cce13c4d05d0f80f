"""Derive the values of cell_2x2_memory.txt: hand-worked 2x2 MDLSTM grids with
memory-state matrices, one hidden unit, one input channel, every cell written
out with scalar math and its own predecessor table per scan direction
(independent of ``oracle/``).

The cell of Section III with the memory-state matrices of Appendix A, in the
reading that both predecessor states c_L (S1) and c_T (S2) enter the input
gate and the two forget gates:
    i   = sig(ln 3  + VI_L c_L + VI_T c_T)
    f_L = sig(-ln 3 + VL_L c_L + VL_T c_T)
    f_T = sig(0     + VT_L c_L + VT_T c_T)
    o   = sig(ln 4)                              (no memory-state input)
    g   = tanh(0.5 x + 0.25 + h_L - 2 h_T)
    c   = i g + f_L c_L + f_T c_T,   h = o tanh(c)
Predecessors outside the grid hand over zeros (Section V, masking).

Usage: python tests/golden/make_cell_2x2_memory.py (the RESULT lines are the
fixture's h and c values, row-major per direction)
"""
from math import exp, log, tanh


def sig(z):
    return 1.0 / (1.0 + exp(-z))


X = {(0, 0): 0.0, (0, 1): 1.0, (1, 0): 2.0, (1, 1): 3.0}
# memory-state weights: rows (i, f_L, f_T), columns (c_L, c_T)
VI_L, VI_T = 0.5, -0.25
VL_L, VL_T = 1.0, 0.5
VT_L, VT_T = -0.75, 0.25


def cell(p, left, top, state):
    hl, cl = state.get(left, (0.0, 0.0))
    ht, ct = state.get(top, (0.0, 0.0))
    i = sig(log(3) + VI_L * cl + VI_T * ct)
    fl = sig(-log(3) + VL_L * cl + VL_T * ct)
    ft = sig(0.0 + VT_L * cl + VT_T * ct)
    o = sig(log(4))
    g = tanh(0.5 * X[p] + 0.25 + 1.0 * hl - 2.0 * ht)
    c = i * g + fl * cl + ft * ct
    h = o * tanh(c)
    state[p] = (h, c)
    print(f"  cell {p}: L={left} T={top} cL={cl:.15f} cT={ct:.15f} i={i:.15f} fL={fl:.15f} fT={ft:.15f} "
          f"g={g:.15f} c={c:.15f} h={h:.15f}")


DIRECTIONS = [
    ([(0, 0), (0, 1), (1, 0), (1, 1)], lambda y, x: (y, x - 1), lambda y, x: (y - 1, x)),  # from top-left
    ([(0, 1), (0, 0), (1, 1), (1, 0)], lambda y, x: (y, x + 1), lambda y, x: (y - 1, x)),  # from top-right
    ([(1, 0), (1, 1), (0, 0), (0, 1)], lambda y, x: (y, x - 1), lambda y, x: (y + 1, x)),  # from bottom-left
    ([(1, 1), (1, 0), (0, 1), (0, 0)], lambda y, x: (y, x + 1), lambda y, x: (y + 1, x)),  # from bottom-right
]

if __name__ == "__main__":
    for d, (order, left_of, top_of) in enumerate(DIRECTIONS):
        print(f"direction {d}")
        st = {}
        for p in order:
            cell(p, left_of(*p), top_of(*p), st)
        print("RESULT", d, " ".join(f"{st[(y, x)][0]:.15e} {st[(y, x)][1]:.15e}" for y in (0, 1) for x in (0, 1)))
