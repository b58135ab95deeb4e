"""Loading the hand-worked fixtures under tests/golden/.

Stored values are closed-form expressions (numbers, + - * /, ln()), so the
fixtures hold the derivation's exact values rather than numbers produced by
either implementation. `ev` evaluates them in float64 and accepts nothing
else.
"""

from __future__ import annotations

import ast
import json
import math
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def ev(expr: str) -> float:
    def go(n):
        if isinstance(n, ast.Constant) and isinstance(n.value, (int, float)):
            return float(n.value)
        if isinstance(n, ast.UnaryOp) and isinstance(n.op, ast.USub):
            return -go(n.operand)
        if isinstance(n, ast.BinOp):
            a, b = go(n.left), go(n.right)
            if isinstance(n.op, ast.Add):
                return a + b
            if isinstance(n.op, ast.Sub):
                return a - b
            if isinstance(n.op, ast.Mult):
                return a * b
            if isinstance(n.op, ast.Div):
                return a / b
        if (isinstance(n, ast.Call) and isinstance(n.func, ast.Name) and n.func.id == "ln"
                and len(n.args) == 1 and not n.keywords):
            return math.log(go(n.args[0]))
        raise ValueError(f"not a closed-form expression: {expr!r}")

    return go(ast.parse(expr, mode="eval").body)


def arr(x) -> np.ndarray:
    """Nested lists of expressions -> float64 array."""
    if isinstance(x, str):
        return np.array(ev(x))
    return np.array([arr(v) for v in x], dtype=np.float64)


def load(name: str) -> dict:
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)
