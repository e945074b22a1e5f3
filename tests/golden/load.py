"""Parser for the hand-worked fixture files in this directory."""
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))


def load_hand_example(name: str = "hand_worked_example.txt"):
    Q, scale, masks, acc, out = [], None, [], [], []
    K = N = None
    with open(os.path.join(HERE, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, *vals = line.split()
            if key == "K":
                K = int(vals[0])
            elif key == "N":
                N = int(vals[0])
            elif key == "Q":
                Q.append([int(v) for v in vals])
            elif key == "scale_hex":
                scale = np.array([int(v, 16) for v in vals], dtype=np.uint32).view(np.float32)
            elif key == "mask_hex":
                masks.append([int(v, 16) for v in vals])
            elif key == "acc":
                acc.append([int(v) for v in vals])
            elif key == "out_hex":
                out.append([int(v, 16) for v in vals])
            else:
                raise ValueError(f"unknown key {key}")
    Q = np.array(Q, dtype=np.int8)
    assert Q.shape == (N, K)
    return dict(
        K=K, N=N,
        W=np.ascontiguousarray(Q.T),  # column-major storage: W[k, n] = Q[n, k]
        scale=scale,
        masks=np.array(masks, dtype=np.uint64),
        acc=np.array(acc, dtype=np.int32),
        out_bits=np.array(out, dtype=np.uint32),
    )


def load_dense_example(name: str = "dense_hand_example.txt"):
    """The hand-worked dense projection example: Q [M, K] int8 row-major,
    scale [M] f32, x [B, K] f32, y [B, M] f64 (exact)."""
    Q, scale, x, y = [], None, [], []
    M = K = None
    with open(os.path.join(HERE, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, *vals = line.split()
            if key == "M":
                M = int(vals[0])
            elif key == "K":
                K = int(vals[0])
            elif key == "Q":
                Q.append([int(v) for v in vals])
            elif key == "scale":
                scale = np.array([float(v) for v in vals], dtype=np.float32)
            elif key == "x":
                x.append([float(v) for v in vals])
            elif key == "y":
                y.append([float(v) for v in vals])
            else:
                raise ValueError(f"unknown key {key}")
    Q = np.array(Q, dtype=np.int8)
    assert Q.shape == (M, K)
    return dict(M=M, K=K, Q=Q, scale=scale, x=np.array(x, dtype=np.float32), y=np.array(y, dtype=np.float64))


def load_quant_example(name: str = "quant_hand_example.txt"):
    """The hand-worked quantizer example: W [M, K] f32, Q [M, K] int8 and the
    scales, with None where the fixture says "floor" (the 1e-8 floor's scale)."""
    W, Q, scale = [], [], None
    M = K = None
    with open(os.path.join(HERE, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, *vals = line.split()
            if key == "M":
                M = int(vals[0])
            elif key == "K":
                K = int(vals[0])
            elif key == "W":
                W.append([float(v) for v in vals])
            elif key == "Q":
                Q.append([int(v) for v in vals])
            elif key == "scale":
                scale = [None if v == "floor" else float(v) for v in vals]
            else:
                raise ValueError(f"unknown key {key}")
    W = np.array(W, dtype=np.float32)
    Q = np.array(Q, dtype=np.int8)
    assert W.shape == Q.shape == (M, K) and len(scale) == M
    return dict(M=M, K=K, W=W, Q=Q, scale=scale)


def load_head_example(name: str = "head_hand_example.txt"):
    """The hand-worked head-verification example: x, xq, Q [V, K], scale,
    approximate logits, candidate order, gap, recomputed logits (per row) and
    (k, threshold, verified, token) cases."""
    d = {"Q": [], "case": []}
    with open(os.path.join(HERE, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, *vals = line.split()
            if key in ("V", "K"):
                d[key] = int(vals[0])
            elif key == "Q":
                d["Q"].append([int(v) for v in vals])
            elif key == "case":
                d["case"].append((int(vals[0]), float(vals[1]), bool(int(vals[2])), int(vals[3])))
            elif key in ("x", "scale", "logits", "gap", "recomputed"):
                d[key] = np.array([float(v) for v in vals], dtype=np.float64)
            elif key in ("xq", "order"):
                d[key] = np.array([int(v) for v in vals], dtype=np.int64)
            else:
                raise ValueError(f"unknown key {key}")
    d["Q"] = np.array(d["Q"], dtype=np.int8)
    d["x"] = d["x"].astype(np.float32)
    d["scale"] = d["scale"].astype(np.float32)
    assert d["Q"].shape == (d["V"], d["K"])
    return d
