"""Reading the hand-worked goldens of tests/golden/ (test helper).

Each file states its citation and derivation; similarities are written as
exact expressions (integers, + - * /, parentheses, sqrt()) that this module
evaluates in fp64 without eval().
"""
from __future__ import annotations

import ast
import json
import math
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def value(s: str) -> float:
    """fp64 value of an exact golden expression."""
    if s.startswith("sqrt1/2"):
        return math.sqrt(0.5)

    def ev(n):
        if isinstance(n, ast.Expression):
            return ev(n.body)
        if isinstance(n, ast.Constant) and isinstance(n.value, (int, float)) and not isinstance(n.value, bool):
            return float(n.value)
        if isinstance(n, ast.UnaryOp) and isinstance(n.op, ast.USub):
            return -ev(n.operand)
        if isinstance(n, ast.BinOp) and type(n.op) in (ast.Add, ast.Sub, ast.Mult, ast.Div):
            a, b = ev(n.left), ev(n.right)
            return {ast.Add: a + b, ast.Sub: a - b, ast.Mult: a * b, ast.Div: a / b if b else math.nan}[type(n.op)]
        if isinstance(n, ast.Call) and isinstance(n.func, ast.Name) and n.func.id == "sqrt" and len(n.args) == 1:
            return math.sqrt(ev(n.args[0]))
        raise ValueError(f"unsupported golden expression {s!r}")

    return ev(ast.parse(s, mode="eval"))


def load(name: str, dtype=np.float64):
    """(golden dict, x [F, N, C]) of a golden file: "tokens" (one frame),
    "frames" ([F][N][C]) or "blocks" ([N][F*C], one position's frames)."""
    g = json.load(open(os.path.join(GOLDEN, name)))
    F, H, W, C = g.get("F", 1), g["H"], g["W"], g["C"]
    if "tokens" in g:
        x = np.array(g["tokens"], dtype=dtype).reshape(1, H * W, C)
    elif "frames" in g:
        x = np.array(g["frames"], dtype=dtype).reshape(F, H * W, C)
    else:
        b = np.array(g["blocks"], dtype=dtype).reshape(H * W, F, C)
        x = np.ascontiguousarray(b.transpose(1, 0, 2))
    return g, x
