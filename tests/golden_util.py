"""Parsing of the hand-worked examples in ``tests/golden/worked_examples.json``."""
import math
from fractions import Fraction

import numpy as np

_NAMES = {"log": math.log, "inf": math.inf, "nan": math.nan, "__builtins__": {}}


def eval_expr(expr: str) -> float:
    return float(eval(expr, {"__builtins__": {}}, dict(_NAMES)))  # fixtures are ours


def frac(s):
    return None if s is None else float(Fraction(s))


def example_arrays(ex, dtype=np.float64):
    """(draft [1,g,V], target [1,g+1,V], tokens [1,g], uniforms [1,g+1])."""
    target = np.array([[eval_expr(e) for e in row] for row in ex["target"]], dtype=np.float64)
    draft = np.array([[eval_expr(e) for e in row] for row in ex["draft"]], dtype=np.float64)
    tokens = np.array(ex["tokens"], dtype=np.int32)[None]
    uniforms = np.array(ex["uniforms"], dtype=np.float64)[None]
    return draft[None].astype(dtype), target[None].astype(dtype), tokens, uniforms
