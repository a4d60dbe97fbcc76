"""Stage a seeded synthetic link-step workload in device memory.

Used by the tests, the smoke check and the benchmark.  Inputs come from
``synth`` (seeded draws, no link-step arithmetic); the plan comes from the
library's own planner; chunk caches are laid into a paged block pool with
physical ids shuffled by the workload seed, so block-table indirection is
exercised.  Nothing here computes any part of the link step.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List

import numpy as np

import synth
from synth.configs import AttnWorkload

from . import epic_link as el


def _bf16_tensor(bits: np.ndarray, device):
    import torch

    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)


@dataclass
class AttnStage:
    wl: AttnWorkload
    cfg: el.epic_attn_cfg
    requests: List[el.Request]
    sizes: el.epic_plan_sizes
    views: Dict[str, np.ndarray]
    dplan: el.DevicePlan
    num_blocks: int
    chunk_block_ids: Dict[int, List[int]]   # chunk id -> physical blocks
    k_cache: object                          # torch bf16 [P, Hkv, 16, D]
    v_cache: object                          # torch bf16 [P, Hkv, D, 16]
    q_s: object
    k_s: object
    v_s: object
    out: object
    lse: object
    workspace: object

    def run(self, stream=None):
        el.epic_link_attention(self.cfg, self.dplan, self.q_s, self.k_s, self.v_s, self.k_cache, self.v_cache,
                               self.out, self.lse, self.workspace, stream)


def chunk_ids(wl: AttnWorkload) -> List[int]:
    seen, order = set(), []
    for r in wl.requests:
        for c in r:
            if c not in seen:
                seen.add(c)
                order.append(c)
    return order


def stage_attention(wl: AttnWorkload, device="cuda", split_blocks: int = 0, spare_blocks: int = 0,
                    threads: int = 8) -> AttnStage:
    """Chunk pool + plan + S-row inputs + output buffers for an attention-level workload."""
    import torch
    from concurrent.futures import ThreadPoolExecutor

    hq, hkv, d = wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    cfg = el.attn_cfg(hq, hkv, d, 0.0, split_blocks)
    ids = chunk_ids(wl)
    nb = {c: -(-wl.chunk_lens[c] // el.BLOCK) for c in ids}
    n_chunk_blocks = sum(nb.values())

    def reqs_with(block_of):
        return [el.Request([wl.chunk_lens[c] for c in r], [block_of[c] for c in r], wl.suffix_lens[i], wl.k)
                for i, r in enumerate(wl.requests)]

    # private blocks needed: plan once with placeholder ids
    placeholder, nxt = {}, 0
    for c in ids:
        placeholder[c] = list(range(nxt, nxt + nb[c]))
        nxt += nb[c]
    n_priv = el.epic_plan_sizes_get(reqs_with(placeholder), cfg, 1 << 30).n_private
    num_blocks = n_chunk_blocks + n_priv + spare_blocks

    perm = np.random.default_rng([wl.seed, 99]).permutation(num_blocks).astype(np.int32)
    block_of, nxt = {}, 0
    for c in ids:
        block_of[c] = perm[nxt:nxt + nb[c]].tolist()
        nxt += nb[c]
    free = perm[nxt:]
    requests = reqs_with(block_of)
    sizes, host, views = el.epic_plan_link(requests, cfg, free, num_blocks)
    dplan = el.DevicePlan(sizes, host, device)

    kpool = np.zeros((num_blocks, hkv, el.BLOCK, d), np.uint16)
    vpool = np.zeros((num_blocks, hkv, d, el.BLOCK), np.uint16)

    def fill(c):
        kr, vr = synth.chunk_cache(wl.seed, c, wl.chunk_lens[c], hkv, d, wl.value_scale, qk_scale=wl.qk_scale)
        kb, vb = el.pack_blocks(kr, vr)
        kpool[block_of[c]] = kb
        vpool[block_of[c]] = vb

    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(fill, ids))
    k_cache = _bf16_tensor(kpool, device)
    v_cache = _bf16_tensor(vpool, device)
    del kpool, vpool

    n_s = sizes.n_s
    q = np.zeros((n_s, hq, d), np.uint16)
    k = np.zeros((n_s, hkv, d), np.uint16)
    v = np.zeros((n_s, hkv, d), np.uint16)
    s_off, s_pos = views["s_off"], views["s_pos"]

    def rows(job):
        r, a, b = job
        q[a:b], k[a:b], v[a:b] = synth.row_qkv(wl.seed, r, s_pos[a:b], hq, hkv, d, wl.value_scale,
                                                wl.qk_scale)

    jobs = []
    for r in range(wl.batch):
        a, b = int(s_off[r]), int(s_off[r + 1])
        step = max(1, (b - a + threads - 1) // threads)
        jobs += [(r, x, min(b, x + step)) for x in range(a, b, step)]
    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(rows, jobs))

    ws_bytes = el.epic_link_workspace_bytes(cfg, sizes)
    return AttnStage(
        wl=wl, cfg=cfg, requests=requests, sizes=sizes, views=views, dplan=dplan, num_blocks=num_blocks,
        chunk_block_ids=block_of, k_cache=k_cache, v_cache=v_cache,
        q_s=_bf16_tensor(q, device), k_s=_bf16_tensor(k, device), v_s=_bf16_tensor(v, device),
        out=torch.zeros((max(1, n_s), hq, d), dtype=torch.bfloat16, device=device),
        lse=torch.zeros((max(1, n_s), hq), dtype=torch.float32, device=device),
        workspace=torch.empty(max(256, ws_bytes), dtype=torch.uint8, device=device),
    )


def attention_flops(views: Dict[str, np.ndarray], hq: int, d: int) -> float:
    """Algorithmic attention flops: 4 * Hq * D * sum over S rows of (position + 1)."""
    return 4.0 * hq * d * float(np.sum(views["s_pos"].astype(np.int64) + 1))
