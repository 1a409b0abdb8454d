"""Readers for the hand-derived fixtures under tests/golden/."""
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _num(tok: str) -> float:
    tok = tok.strip()
    if tok.lower().lstrip("+-").startswith("0x"):
        return float.fromhex(tok)
    return float(tok)


def _records(name: str, opener: str):
    rec = None
    with open(os.path.join(GOLDEN, name)) as f:
        for raw in f:
            line = raw.split("#", 1)[0].strip()
            if not line:
                continue
            key, _, rest = line.partition(" ")
            if key == opener:
                rec = {"name": rest.strip(), "_lines": []}
            elif key == "end":
                yield rec
                rec = None
            else:
                rec["_lines"].append((key, rest.split()))


def sqnorm_cases():
    """Yields (name, [(numel, {index: value})], expect_sk list, expect_s)."""
    for rec in _records("sqnorm_order.txt", "case"):
        tensors, sk, s = [], None, None
        for key, toks in rec["_lines"]:
            if key == "tensor":
                n = int(toks[0])
                vals = {}
                for t in toks[1:]:
                    idx, _, v = t.partition("=")
                    if ".." in idx:
                        lo, hi = (int(x) for x in idx.split(".."))
                        for i in range(lo, hi + 1):
                            vals[i] = _num(v)
                    else:
                        vals[int(idx)] = _num(v)
                tensors.append((n, vals))
            elif key == "expect_sk":
                sk = [_num(t) for t in toks]
            elif key == "expect_s":
                s = _num(toks[0])
        yield rec["name"], tensors, sk, s


def adamw_examples(name: str = "adamw8_worked_examples.txt"):
    """Yields dicts with scalar hyperparameters and numpy arrays."""
    ints = {"m_codes": np.int8, "v_codes": np.uint8, "expect_m_codes": np.int8,
            "expect_v_codes": np.uint8}
    for rec in _records(name, "example"):
        ex = {"name": rec["name"]}
        for key, toks in rec["_lines"]:
            if key in ("block_size", "t"):
                ex[key] = int(toks[0])
            elif key in ("lr", "beta1", "beta2", "eps", "weight_decay", "coef"):
                ex[key] = _num(toks[0])
            elif key in ints:
                ex[key] = np.array([int(t) for t in toks], dtype=ints[key])
            else:
                ex[key] = np.array([_num(t) for t in toks], dtype=np.float32)
        yield ex


def dense(n: int, vals: dict, dtype=np.float32) -> np.ndarray:
    x = np.zeros(n, dtype=np.float32)
    for i, v in vals.items():
        x[i] = v
    return x.astype(dtype)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16, returned as raw uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
