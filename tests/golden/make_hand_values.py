"""Write hand_values.json: two-point inputs whose reductions have short closed forms.

The paper prints no worked numeric example, so each value here is the formula
it cites evaluated by hand on inputs chosen so the result is a closed form;
only the standard library's math module is used.  Run from the repo root:
    python tests/golden/make_hand_values.py
"""
import json
import math
import os

E = math.exp

VALUES = {
    "_about": "Hand-derived values of the reductions on two-point inputs. The paper prints no "
              "worked example; each entry states the inputs, the formula it evaluates and the "
              "closed form used. Written by make_hand_values.py.",
    "gauss_two_point": {
        "cite": "Eq. (1)", "x": [[0, 0, 0]], "y": [[0, 0, 0], [1, 0, 0]], "b": [[1], [2]],
        "sigma": 1.0, "closed_form": "1*exp(0) + 2*exp(-1/2)", "value": 1 + 2 * E(-0.5)},
    "gauss_two_point_scaled": {
        "cite": "Eq. (1)", "x": [[0.5, -1, 2]], "y": [[0.5, -1, 2], [0.5, -1, 2.25]],
        "b": [[3], [-1]], "sigma": 0.125,
        "closed_form": "3*exp(0) - exp(-(1/4)^2 / (2 (1/8)^2)) = 3 - exp(-2)", "value": 3 - E(-2.0)},
    "laplace_two_point": {
        "cite": "Eq. (2) with F = exp(-|x-y|/sigma) b", "x": [[0, 0, 0]],
        "y": [[0, 0, 0], [3, 4, 0]], "b": [[1], [2]], "sigma": 5.0,
        "closed_form": "1 + 2*exp(-5/5)", "value": 1 + 2 * E(-1.0)},
    "sqdist_two_point": {
        "cite": "Eq. (2) with F = |x-y|^2 b", "x": [[1, 2, 3]], "y": [[0, 0, 0], [1, 2, 4]],
        "b": [[1], [10]], "sigma": 1.0, "closed_form": "14*1 + 1*10", "value": 24.0},
    "gradx_one_point": {
        "cite": "Sec. 2 (Backpropagation): d/dx_i of Eq. (1)", "x": [[0, 0, 0]], "y": [[1, 2, 0]],
        "b": [[2]], "sigma": 2.0,
        "closed_form": "a = 2 exp(-5/8); g = a (y - x) / sigma^2 = a (1, 2, 0) / 4",
        "value": [2 * E(-5 / 8), 2 * E(-5 / 8) / 4, 2 * E(-5 / 8) * 2 / 4, 0.0]},
    "vjp_two_point": {
        "cite": "Sec. 2 (Backpropagation): d/dx_i of L = sum_i <e_i, a_i>, a_i from Eq. (1) with E = 2",
        "x": [[0, 0]], "y": [[1, 0], [0, 2]], "b": [[1, 2], [-1, 0]], "e": [[3, 1]], "sigma": 1.0,
        "closed_form": "<e, b_0> = 5, <e, b_1> = -3; g = 5 exp(-1/2) (1, 0) - 3 exp(-2) (0, 2)",
        "value": [5 * E(-0.5), -6 * E(-2.0)]},
    "extreme_small": {
        "cite": "Sec. 2 (.min(), .max(), .argmin()): extreme entries of a row of F and their lowest index",
        "x": [[0, 0]], "y": [[2, 0], [1, 0], [0, 1], [0, 0], [-1, 0], [3, 3]],
        "b": [[1], [2], [-2], [0.5], [2], [7]], "sigma": 1.0,
        "closed_form": "squared distances (4, 1, 1, 0, 1, 18): min 0 at j=3, max 18 at j=5; Gaussian "
                       "F = exp(-d/2) b = (e^-2, 2e^-1/2, -2e^-1/2, 1/2, 2e^-1/2, 7e^-9): max 2e^-1/2 "
                       "at j=1 (tie with j=4 keeps the lower index), min -2e^-1/2 at j=2",
        "value": {"sqdist_min": [0.0, 3], "sqdist_max": [18.0, 5],
                  "gauss_max": [2 * E(-0.5), 1], "gauss_min": [-2 * E(-0.5), 2]}},
    "lse_two_point": {
        "cite": "Eq. (2) with the log-sum-exp reduction of Sec. 2, F = g_j - |x-y|^2/eps",
        "x": [[0, 0]], "y": [[0, 0], [1, 1]], "g": [[0], [2]], "eps": 1.0,
        "closed_form": "log(exp(0 - 0) + exp(2 - 2)) = log 2", "value": math.log(2.0)},
    "argkmin_small": {
        "cite": "Sec. 2 (argKmin): indices of the K smallest entries of a row", "x": [[0, 0]],
        "y": [[2, 0], [1, 0], [0, 1], [0, 0], [-1, 0], [3, 3]], "K": 4,
        "closed_form": "squared distances (4, 1, 1, 0, 1, 18): j=3 (0), then the three ties at 1 "
                       "by index: 1, 2, 4", "value": [3, 1, 2, 4]},
}

if __name__ == "__main__":
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "hand_values.json")
    with open(path, "w") as f:
        json.dump(VALUES, f, indent=1)
        f.write("\n")
    print("wrote", path)
