"""Reader for the hand-derived worked examples under tests/golden/."""
import glob
import os

import numpy as np

GOLDEN_DIR = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
MODES = {"projected": 0, "sliced": 1, "full": 2}


def load(path):
    spec = {}
    rows = {"V": {}, "K": {}, "alpha": {}, "H": {}}
    with open(path) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            lhs, rhs = (s.strip() for s in line.split("=", 1))
            key = lhs.split()
            if key[0] == "mode":
                spec["mode"] = MODES[rhs]
                continue
            nums = [float(x) for x in rhs.split()]
            if key[0] in ("V", "K"):
                rows[key[0]][(int(key[1]), int(key[2]))] = nums
            elif key[0] in ("alpha", "H"):
                rows[key[0]][int(key[1])] = nums
            elif key[0] == "q":
                spec["q"] = np.array(nums)
            else:
                spec[key[0]] = nums[0]
    S, N, d, r = (int(spec[k]) for k in ("S", "N", "d", "r"))
    V = np.zeros((S, N, d))
    for (i, n), v in rows["V"].items():
        V[i, n] = v
    K = None
    if rows["K"]:
        K = np.zeros((S, N, r))
        for (i, n), v in rows["K"].items():
            K[i, n] = v
    alpha = np.array([rows["alpha"][n] for n in range(N)])
    H = np.array([rows["H"][n] for n in range(N)])
    return dict(mode=spec["mode"], S=S, N=N, d=d, r=r, eps=spec["eps"], q=spec["q"],
                V=V, K=K, alpha=alpha, H=H, name=os.path.basename(path))


def all_fixtures():
    """The single-site routing examples (files named after a key mode)."""
    names = sorted(glob.glob(os.path.join(GOLDEN_DIR, "*.txt")))
    return [load(p) for p in names
            if os.path.basename(p).split("_")[0] in ("sliced", "projected", "full")]


def load_block(name):
    """A block-source worked example: outputs O[i], block size c, site t."""
    spec, O, res = {}, {}, {}
    with open(os.path.join(GOLDEN_DIR, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            lhs, rhs = (x.strip() for x in line.split("=", 1))
            key = lhs.split()
            nums = [float(x) for x in rhs.split()]
            if key[0] == "O":
                O[int(key[1])] = nums
            elif key[0] in ("alpha", "H", "q"):
                res[key[0]] = np.array(nums)
            else:
                spec[key[0]] = nums[0]
    t = int(spec["t"])
    return dict(t=t, c=int(spec["c"]), d=int(spec["d"]), r=int(spec["r"]), eps=spec["eps"],
                O=np.array([O[i] for i in range(t)])[:, None, :], **res)


def load_table1():
    """Rows (kind, blocks, rank, printed value) of the Table 1 fixture."""
    rows = []
    with open(os.path.join(GOLDEN_DIR, "table1_added_flops.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                kind, nb, r, v = line.split()
                rows.append((kind, int(nb), int(r), float(v)))
    return rows
