"""Placing a generated workload's values into a Session's device buffers.

Only data placement: cached unit states are copied into their pool pages
(token j of a unit in block j // B at slot j % B, page layout [H_kv][B][d]),
and fresh per-token projections are laid out as [T][H][d] in the plan's row
order (the order tsr_plan_compute_positions reports).
"""
from __future__ import annotations

import numpy as np
import torch


def _pages_from_tokens(x: np.ndarray, page_size: int) -> np.ndarray:
    """[n][H][d] -> [ceil(n/B)][H][B][d], zero-padded past n."""
    n, H, d = x.shape
    npg = -(-n // page_size)
    pad = np.zeros((npg * page_size, H, d), dtype=x.dtype)
    pad[:n] = x
    return np.ascontiguousarray(pad.reshape(npg, page_size, H, d).transpose(0, 2, 1, 3))


def upload_pool(sess, wl, unit_ids=None, layer: int = 0) -> None:
    """Write the cached state of every unit in `unit_ids` (default: every unit
    that is a HIT somewhere in the batch) into its pool pages."""
    B = wl.model.page_size
    ids = wl.hit_unit_ids() if unit_ids is None else unit_ids
    for uid in ids:
        dev = sess.pool_k.device          # the GPU, or the host for a host-tier pool
        pages = torch.as_tensor(np.asarray(wl.unit_pages[uid], dtype=np.int64), device=dev)
        if sess.e4m3:
            k, v, ks, vs = wl.unit_state_e4m3(uid)
            sc = torch.from_numpy(np.stack([ks, vs], axis=1)).to(dev)
            sess.pool_scale[layer][pages] = sc
        else:
            k, v = wl.unit_state(uid)
        for src, dst in ((k, sess.pool_k[layer]), (v, sess.pool_v[layer])):
            t = torch.from_numpy(_pages_from_tokens(src, B)).to(dev)
            dst[pages] = t.to(dst.dtype)


def fresh_inputs(sess, wl, plan):
    """q, k, v [T][H][d] (act dtype, device) for the plan's computed rows."""
    pos, req = plan.compute_positions()
    m = wl.model
    T = len(pos)
    q = np.empty((T, m.n_q_heads, m.head_dim), dtype=np.float32)
    k = np.empty((T, m.n_kv_heads, m.head_dim), dtype=np.float32)
    v = np.empty_like(k)
    for r in np.unique(req):
        rows = np.nonzero(req == r)[0]
        q[rows], k[rows], v[rows] = wl.fresh(int(r), pos[rows])
    to = lambda a: torch.from_numpy(a).to(sess.device).to(sess.act_dtype)
    return to(q), to(k), to(v)


def request_kv(sess, wl, r: int, layer: int = 0):
    """Assembled K, V of request r from the request pages, [P][H_kv][d] on the
    host: fp32 values, or for e4m3 arenas (codes_k, codes_v, scale_k[P],
    scale_v[P]) with each position's page scale."""
    req = wl.requests[r]
    B = wl.model.page_size
    bt = torch.as_tensor(np.asarray(req.block_table, dtype=np.int64), device=sess.device)
    out = []
    for arena in (sess.req_k[layer], sess.req_v[layer]):
        pages = arena[bt]                                   # [npg][H][B][d]
        dense = pages.permute(0, 2, 1, 3).reshape(-1, *pages.shape[1:2], pages.shape[-1])
        dense = dense[:req.prompt_len]
        out.append(dense.cpu().numpy() if sess.e4m3 else dense.float().cpu().numpy())
    if not sess.e4m3:
        return out[0], out[1]
    sc = sess.req_scale[layer][bt].cpu().numpy()            # [npg][2]
    per_pos = np.repeat(sc, B, axis=0)[:req.prompt_len]
    return out[0], out[1], per_pos[:, 0].copy(), per_pos[:, 1].copy()
