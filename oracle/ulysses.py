"""Local halves of the Ulysses exchange as pure index maps (numpy).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py): never imported by the
product path.

Background, Sequence Parallelism: before attention an all-to-all turns the
sequence-sharded layout (each GPU holds n = L/sp tokens of a sequence, all
H heads) into the head-sharded layout (each GPU holds all L tokens for a
subset of heads); a second all-to-all after attention restores it.  On one
GPU the exchange is the identity, so what remains is the sender-side
permutation, laid out where the exchange would land each chunk:

  per item j with n = L_j / sp_j, kind head count H (Hq or Hkv),
  H_loc = H / sp if H >= sp else 1, and head(s, h') = s*H_loc + h'
  (H >= sp) or floor(s*H/sp) (H < sp, the KV head is replicated):

  seq layout  : item j at token offset c_j = sum_{i<j} L_i / sp_i, [n, H, D]
  head layout : item j at element offset D * sum_{i<j} L_i * H_loc(i), [L_j, H_loc, D]

  pack   : X_head[j][s*n + t, h', :] = X_seq[c_j + t, head(s, h'), :]
  unpack : the inverse for H >= sp; for H < sp, KV head g collects replicas
           s with head(s, 0) = g:
             SELECT: X_seq[c_j + t, g] = X_head[j][s_g*n + t, 0], s_g = g*sp/H
             SUM:    X_seq[c_j + t, g] = round(sum over those s, in increasing
                     s, of float32(X_head[j][s*n + t, 0]))  (float32 adds; the
                     result rounded to bf16 to nearest even for bf16 data;
                     float64 data -- reference values, not a stored format --
                     is summed in float64, without rounding)

Arrays are raw element arrays (uint16 for bf16, float32 for f32); pack and
SELECT move bits only.
"""
from __future__ import annotations

import numpy as np

__all__ = ["h_loc", "replica_heads", "pack", "unpack"]


def h_loc(H: int, sp: int) -> int:
    return H // sp if H >= sp else 1


def replica_heads(H: int, sp: int):
    """head(s, 0) for each destination block s (H < sp: replicated KV heads)."""
    return [(s * H) // sp for s in range(sp)]


def _round_f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


def _seq_offsets(lengths, sp):
    c, out = 0, []
    for L, s in zip(lengths, sp):
        out.append(c)
        c += L // s
    return out, c


def _head_offsets(lengths, sp, H, D):
    e, out = 0, []
    for L, s in zip(lengths, sp):
        out.append(e)
        e += L * h_loc(H, s) * D
    return out, e


def pack(x_seq, lengths, sp, H, D):
    """Sequence-sharded -> head-sharded layout (flat element arrays)."""
    lengths = [int(a) for a in lengths]
    sp = [int(a) for a in sp]
    c_off, T = _seq_offsets(lengths, sp)
    e_off, E = _head_offsets(lengths, sp, H, D)
    xs = np.asarray(x_seq).reshape(T, H, D)
    out = np.empty(E, dtype=xs.dtype)
    for j, (L, s) in enumerate(zip(lengths, sp)):
        n, hl = L // s, h_loc(H, s)
        blk = xs[c_off[j]:c_off[j] + n]                      # [n, H, D]
        if H >= s:
            y = blk.reshape(n, s, hl, D).transpose(1, 0, 2, 3)   # [s, n, hl, D]
        else:
            y = blk[:, replica_heads(H, s), :].transpose(1, 0, 2)[:, :, None, :]
        out[e_off[j]:e_off[j] + L * hl * D] = y.reshape(-1)
    return out


def unpack(x_head, lengths, sp, H, D, mode="select"):
    """Head-sharded -> sequence-sharded layout.  mode: 'select' or 'sum'."""
    lengths = [int(a) for a in lengths]
    sp = [int(a) for a in sp]
    c_off, T = _seq_offsets(lengths, sp)
    e_off, _ = _head_offsets(lengths, sp, H, D)
    xh = np.asarray(x_head)
    out = np.empty((T, H, D), dtype=xh.dtype)
    for j, (L, s) in enumerate(zip(lengths, sp)):
        n, hl = L // s, h_loc(H, s)
        y = xh[e_off[j]:e_off[j] + L * hl * D].reshape(s, n, hl, D)
        dst = out[c_off[j]:c_off[j] + n]
        if H >= s:
            dst[:] = y.transpose(1, 0, 2, 3).reshape(n, H, D)
            continue
        reps = s // H
        for g in range(H):
            if mode == "select":
                dst[:, g, :] = y[g * reps, :, 0, :]
            elif mode == "sum":
                if xh.dtype == np.uint16:
                    acc = (y[g * reps, :, 0, :].astype(np.uint32) << np.uint32(16)).view(np.float32).copy()
                    for r in range(1, reps):
                        acc = acc + (y[g * reps + r, :, 0, :].astype(np.uint32) << np.uint32(16)).view(np.float32)
                    dst[:, g, :] = _round_f32_to_bf16_bits(acc)
                elif xh.dtype == np.float64:
                    acc = y[g * reps, :, 0, :].copy()
                    for r in range(1, reps):
                        acc = acc + y[g * reps + r, :, 0, :]
                    dst[:, g, :] = acc
                else:
                    acc = y[g * reps, :, 0, :].astype(np.float32)
                    for r in range(1, reps):
                        acc = acc + y[g * reps + r, :, 0, :].astype(np.float32)
                    dst[:, g, :] = acc
            else:
                raise ValueError(mode)
    return out.reshape(-1)
