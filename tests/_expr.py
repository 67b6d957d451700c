"""Tiny evaluator for the hand-written golden fixtures: numbers, + - * /, ln(), exp()."""
import ast
import math
from fractions import Fraction

_FUNCS = {"ln": math.log, "exp": math.exp}


def value(expr) -> float:
    if isinstance(expr, (int, float)):
        return float(expr)
    node = ast.parse(str(expr), mode="eval").body
    return float(_eval(node))


def _eval(n):
    if isinstance(n, ast.Constant) and isinstance(n.value, (int, float)):
        return Fraction(n.value) if isinstance(n.value, int) else n.value
    if isinstance(n, ast.UnaryOp) and isinstance(n.op, ast.USub):
        return -_eval(n.operand)
    if isinstance(n, ast.BinOp):
        a, b = _eval(n.left), _eval(n.right)
        if isinstance(n.op, ast.Add):
            return a + b
        if isinstance(n.op, ast.Sub):
            return a - b
        if isinstance(n.op, ast.Mult):
            return a * b
        if isinstance(n.op, ast.Div):
            return a / b
    if isinstance(n, ast.Call) and isinstance(n.func, ast.Name) and n.func.id in _FUNCS:
        (arg,) = n.args
        return _FUNCS[n.func.id](float(_eval(arg)))
    raise ValueError(f"unsupported expression: {ast.dump(n)}")
