"""Loader of tests/golden/worked_example.json: the hand-worked example whose
expected values are closed forms written as arithmetic expressions (numbers,
+ - * /, parentheses and ln(x)); this module evaluates them, nothing else."""
import ast
import json
import math
import os

PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "worked_example.json")
MODES = {"STANDARD": 0, "CM": 1, "GREEDY": 2}


def value(expr) -> float:
    """A closed form of the fixture: a number, '-inf'/'inf', or an expression."""
    if isinstance(expr, (int, float)):
        return float(expr)
    if expr in ("-inf", "inf"):
        return float(expr)

    def ev(n):
        if isinstance(n, ast.Expression):
            return ev(n.body)
        if isinstance(n, ast.Constant) and isinstance(n.value, (int, float)):
            return float(n.value)
        if isinstance(n, ast.UnaryOp) and isinstance(n.op, ast.USub):
            return -ev(n.operand)
        if isinstance(n, ast.BinOp) and isinstance(n.op, (ast.Add, ast.Sub, ast.Mult, ast.Div)):
            a, b = ev(n.left), ev(n.right)
            return {ast.Add: a + b, ast.Sub: a - b, ast.Mult: a * b}.get(type(n.op), a / b if b else math.nan)
        if isinstance(n, ast.Call) and isinstance(n.func, ast.Name) and n.func.id == "ln" and len(n.args) == 1:
            return math.log(ev(n.args[0]))
        raise ValueError(f"not a closed form of the fixture: {expr!r}")

    return ev(ast.parse(expr, mode="eval"))


def load() -> dict:
    with open(PATH) as f:
        fx = json.load(f)
    fx["drafter_z"] = [[value(x) for x in r["z"]] for r in fx["drafter_rows"]]
    fx["target_z"] = [[value(x) for x in r] for r in fx["verify"]["target_rows"]]
    return fx
