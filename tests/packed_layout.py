"""The packed operand layout of include/micromix.h, written out in numpy for
the tests: tile() turns row-major codes and scales (the oracle's form) into
the four packed buffers, zero padding included, and untile() reverses it.

Only a layout transform: it touches no value, so the parity tests can compare
the GPU's buffers with the oracle's output byte for byte.
"""

from __future__ import annotations

import numpy as np

ROW_GROUP = 32
STEP_BLOCKS = 4
STEP_ROW_BYTES = (64, 96, 128)  # E2M1, E3M2, E4M3
BLOCK_BYTES = (16, 24, 32)


def geometry(rows: int, split) -> dict:
    rp = -(-rows // ROW_GROUP) * ROW_GROUP
    nb = [int(p) // 32 for p in split]
    steps = [-(-n // STEP_BLOCKS) for n in nb]
    return {"rp": rp, "nb": nb, "steps": steps,
            "bytes": [steps[g] * rp * STEP_ROW_BYTES[g] for g in range(3)] + [sum(steps) * rp * STEP_BLOCKS]}


def _codes_to_blocks(rowmajor: np.ndarray, g: int, rows: int, rp: int, nb: int, steps: int) -> np.ndarray:
    """[rows, nb * block_bytes] -> [rp, steps, 4, block_bytes] with zero padding."""
    bb = BLOCK_BYTES[g]
    out = np.zeros((rp, steps * STEP_BLOCKS, bb), np.uint8)
    out[:rows, :nb] = np.asarray(rowmajor, np.uint8).reshape(rows, nb, bb)
    return out.reshape(rp, steps, STEP_BLOCKS, bb)


def tile(q4, q6, q8, sc, rows: int, split) -> dict:
    """Packed buffers from row-major packed codes ([rows, p/2], [rows, 3p/4],
    [rows, p]) and scales ([rows, K/32], E2M1 blocks first)."""
    geo = geometry(rows, split)
    rp, nb, steps = geo["rp"], geo["nb"], geo["steps"]
    out = {}
    for g, (name, arr) in enumerate((("q4", q4), ("q6", q6), ("q8", q8))):
        if steps[g] == 0:
            out[name] = np.zeros(0, np.uint8)
            continue
        blk = _codes_to_blocks(arr, g, rows, rp, nb[g], steps[g])  # [rp, S, 4, bb]
        blk = blk.reshape(rp // ROW_GROUP, ROW_GROUP, steps[g], STEP_BLOCKS, BLOCK_BYTES[g])
        if g == 2:  # block j of row r: halves at slots 2j, 2j+1 of 512 bytes each
            blk = blk.reshape(rp // ROW_GROUP, ROW_GROUP, steps[g], STEP_BLOCKS, 2, 16)
            rec = blk.transpose(2, 0, 3, 4, 1, 5)  # [S, q, j, h, r, 16]
        else:  # [S, q, j, r, bb]
            rec = blk.transpose(2, 0, 3, 1, 4)
        out[name] = np.ascontiguousarray(rec).reshape(-1)
    # scales: [T, rp, 4]
    sc = np.asarray(sc, np.uint8)
    parts, b0 = [], 0
    for g in range(3):
        s = np.zeros((rp, steps[g] * STEP_BLOCKS), np.uint8)
        s[:rows, :nb[g]] = sc[:, b0:b0 + nb[g]]
        b0 += nb[g]
        parts.append(s.reshape(rp, steps[g], STEP_BLOCKS).transpose(1, 0, 2))
    out["sc"] = np.ascontiguousarray(np.concatenate(parts, axis=0)).reshape(-1)
    return out


def untile(raw: dict, rows: int, split) -> dict:
    """Row-major q4 / q6 / q8 / sc (the oracle's form) from packed buffers."""
    geo = geometry(rows, split)
    rp, nb, steps = geo["rp"], geo["nb"], geo["steps"]
    out = {}
    for g, name in enumerate(("q4", "q6", "q8")):
        bb = BLOCK_BYTES[g]
        if steps[g] == 0:
            out[name] = np.zeros((rows, 0), np.uint8)
            continue
        buf = np.asarray(raw[name], np.uint8)[: geo["bytes"][g]]
        if g == 2:
            rec = buf.reshape(steps[g], rp // ROW_GROUP, STEP_BLOCKS, 2, ROW_GROUP, 16)
            blk = rec.transpose(1, 4, 0, 2, 3, 5)  # [q, r, S, j, h, 16]
        else:
            rec = buf.reshape(steps[g], rp // ROW_GROUP, STEP_BLOCKS, ROW_GROUP, bb)
            blk = rec.transpose(1, 3, 0, 2, 4)  # [q, r, S, j, bb]
        blk = np.ascontiguousarray(blk).reshape(rp, steps[g] * STEP_BLOCKS * bb)
        out[name] = blk[:rows, : nb[g] * bb]
    scb = np.asarray(raw["sc"], np.uint8)[: geo["bytes"][3]].reshape(sum(steps), rp, STEP_BLOCKS)
    cols, t0 = [], 0
    for g in range(3):
        s = scb[t0:t0 + steps[g]].transpose(1, 0, 2).reshape(rp, steps[g] * STEP_BLOCKS)
        cols.append(s[:rows, : nb[g]])
        t0 += steps[g]
    out["sc"] = np.concatenate(cols, axis=1)
    return out
