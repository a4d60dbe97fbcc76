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
    spare: List[int] = None                  # free blocks the link plan did not take

    def run(self, stream=None):
        el.epic_link_attention(self.cfg, self.dplan, self.q_s, self.k_s, self.v_s, self.k_cache, self.v_cache,
                               self.out, self.lse, self.workspace, stream)


@dataclass
class DecodeStage:
    """One decode step after a link (or decode) plan: the new tokens' rows and plan."""
    cfg: el.epic_attn_cfg
    sizes: el.epic_plan_sizes
    views: Dict[str, np.ndarray]
    dplan: el.DevicePlan
    spare: List[int]                         # free blocks left after this step
    q_s: object
    k_s: object
    v_s: object
    out: object
    lse: object
    workspace: object

    def run(self, k_cache, v_cache, stream=None):
        el.epic_link_attention(self.cfg, self.dplan, self.q_s, self.k_s, self.v_s, k_cache, v_cache,
                               self.out, self.lse, self.workspace, stream)


def stage_decode(wl: AttnWorkload, cfg: el.epic_attn_cfg, prev_sizes: el.epic_plan_sizes, prev_host: np.ndarray,
                 spare: List[int], num_blocks: int, new_tokens: List[int], device="cuda") -> DecodeStage:
    """Decode plan appending new_tokens[r] tokens to request r of the previous plan, with
    the new tokens' q / k / v drawn by position like the link step's rows."""
    import torch

    hq, hkv, d = wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    sizes, host, views = el.epic_plan_decode(prev_sizes, prev_host, new_tokens, cfg, spare, num_blocks)
    taken = sizes.n_linked_blocks - prev_sizes.n_linked_blocks
    n_s = sizes.n_s
    q = np.zeros((max(1, n_s), hq, d), np.uint16)
    k = np.zeros((max(1, n_s), hkv, d), np.uint16)
    v = np.zeros((max(1, n_s), hkv, d), np.uint16)
    for r in range(sizes.batch):
        a, b = int(views["s_off"][r]), int(views["s_off"][r + 1])
        if b > a:
            q[a:b], k[a:b], v[a:b] = synth.row_qkv(wl.seed, r, views["s_pos"][a:b], hq, hkv, d, wl.value_scale,
                                                    wl.qk_scale)
    ws_bytes = el.epic_link_workspace_bytes(cfg, sizes)
    return DecodeStage(
        cfg=cfg, sizes=sizes, views=views, dplan=el.DevicePlan(sizes, host, device), spare=list(spare[taken:]),
        q_s=_bf16_tensor(q, device), k_s=_bf16_tensor(k, device), v_s=_bf16_tensor(v, device),
        out=torch.zeros((max(1, n_s), hq, d), dtype=torch.bfloat16, device=device),
        lse=torch.zeros((max(1, n_s), hq), dtype=torch.float32, device=device),
        workspace=torch.empty(max(256, ws_bytes), dtype=torch.uint8, device=device),
    )


def chunk_ids(wl: AttnWorkload) -> List[int]:
    seen, order = set(), []
    for r in wl.requests:
        for c in r:
            if c not in seen:
                seen.add(c)
                order.append(c)
    return order


def stage_attention(wl: AttnWorkload, device="cuda", split_blocks: int = 0, spare_blocks: int = 0,
                    threads: int = 8, tile_rows: int = 0, rerotate_theta: float = 0.0) -> AttnStage:
    """Chunk pool + plan + S-row inputs + output buffers for an attention-level workload.
    rerotate_theta > 0: the re-rotation variant (cached K of chunks 1.. moved to its
    linked positions, rotary base rerotate_theta)."""
    import torch
    from concurrent.futures import ThreadPoolExecutor

    hq, hkv, d = wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    cfg = el.attn_cfg(hq, hkv, d, 0.0, split_blocks, tile_rows, rerotate_theta)
    rerotate = rerotate_theta > 0
    ids = chunk_ids(wl)
    nb = {c: -(-wl.chunk_lens[c] // el.BLOCK) for c in ids}
    n_chunk_blocks = sum(nb.values())

    def reqs_with(block_of):
        return [el.Request([wl.chunk_lens[c] for c in r], [block_of[c] for c in r], wl.suffix_lens[i], wl.k,
                           rerotate) for i, r in enumerate(wl.requests)]

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
        spare=[int(x) for x in free[sizes.n_private:]],
    )


def attention_flops(views: Dict[str, np.ndarray], hq: int, d: int) -> float:
    """Algorithmic attention flops: 4 * Hq * D * sum over S rows of (position + 1)."""
    return 4.0 * hq * d * float(np.sum(views["s_pos"].astype(np.int64) + 1))


# ---------------------------------------------------------------- model level

@dataclass
class ModelStage:
    wl: object
    cfg: el.epic_model_cfg
    weights: List[Dict[str, object]]         # per layer: torch bf16 tensors
    layers: List[el.epic_layer_weights]
    final_norm: object
    k_caches: List[object]                   # per layer: torch bf16 [P, Hkv, 16, D]
    v_caches: List[object]                   # per layer: torch bf16 [P, Hkv, D, 16]
    requests: List[el.Request]
    chunk_block_ids: List[List[int]]
    sizes: el.epic_plan_sizes
    views: Dict[str, np.ndarray]
    dplan: el.DevicePlan
    emb: object                              # torch fp32 [n_s, hidden]: layer-0 rows of S
    hidden: object                           # torch fp32 [n_s, hidden], overwritten by a run
    out: object                              # torch fp32 [n_s, hidden]
    workspace: object
    compile_stage: object = None             # kept with keep_compile=True (its out: compiled hidden rows)

    def run(self, stream=None):
        self.hidden.copy_(self.emb)
        el.epic_link_model(self.cfg, self.layers, self.final_norm, self.dplan, self.hidden, self.k_caches,
                           self.v_caches, self.out, self.workspace, stream)


def model_cfg(wl, n_layers: int, tile_rows: int = 0, split_blocks: int = 0) -> el.epic_model_cfg:
    return el.epic_model_cfg(el.attn_cfg(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, split_blocks=split_blocks,
                                         tile_rows=tile_rows), wl.hidden, wl.ffn, n_layers, wl.rope_theta, wl.rms_eps)


def _tok_rows(wl, chunk_ids_of_req, chunk_lens, suffix_len, positions, req=0):
    """Embeddings of the tokens at the given linked positions of one request."""
    offs = np.cumsum([0] + list(chunk_lens))
    out = np.empty((len(positions), wl.hidden), np.float32)
    for i, p in enumerate(positions):
        j = int(np.searchsorted(offs, p, side="right") - 1)
        if j < len(chunk_lens):
            out[i] = synth.token_embeddings(wl.seed, 0, chunk_ids_of_req[j], [p - offs[j]], wl.hidden)[0]
        else:
            out[i] = synth.token_embeddings(wl.seed, 1, req, [p - offs[-1]], wl.hidden)[0]
    return out


def _device_weights(wl, layer: int, device):
    """Random-init weights drawn on the device (seeded torch generator), same shapes and
    distributions as synth.model_weights; for timing runs, where the values do not matter."""
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(wl.seed * 1000 + layer)
    hq, hkv, d, H, F = wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.hidden, wl.ffn

    def lin(out_f, in_f):
        return (torch.randn(out_f, in_f, generator=gen, device=device) * (0.5 / in_f ** 0.5)).to(torch.bfloat16)

    def norm(n):
        return (1.0 + 0.1 * torch.randn(n, generator=gen, device=device)).to(torch.bfloat16)

    return {"attn_norm": norm(H), "wqkv": lin((hq + 2 * hkv) * d, H), "wo": lin(H, hq * d), "mlp_norm": norm(H),
            "w_gate_up": lin(2 * F, H), "w_down": lin(H, F)}


@dataclass
class CompileStage:
    """Compile step of a model-level workload: every chunk prefilled alone (after
    n_dummy dummy tokens for LegoLink-0), its K/V stored into its chunk blocks."""

    cfg: el.epic_model_cfg
    layers: List[el.epic_layer_weights]
    final_norm: object
    sizes: el.epic_plan_sizes
    views: Dict[str, np.ndarray]
    dplan: el.DevicePlan
    emb: object                              # torch fp32 [n_s, hidden]: per chunk, dummies then tokens
    hidden: object
    out: object
    workspace: object

    def run(self, k_caches, v_caches, stream=None):
        self.hidden.copy_(self.emb)
        el.epic_link_model(self.cfg, self.layers, self.final_norm, self.dplan, self.hidden, k_caches, v_caches,
                           self.out, self.workspace, stream)


def compile_rows(wl, n_dummy: int) -> np.ndarray:
    """Layer-0 rows of the compile plan: for every chunk, n_dummy dummy rows, then its tokens."""
    H = wl.hidden
    dummy = synth.dummy_embeddings(wl.seed, n_dummy, H)
    parts = []
    for j, n in enumerate(wl.chunk_lens):
        if n_dummy:
            parts.append(dummy)
        parts.append(synth.token_embeddings(wl.seed, 0, j, range(n), H))
    return np.concatenate(parts)


def stage_compile(wl, cfg, layers, final_norm, chunk_blocks, free, num_blocks, n_dummy, device="cuda"):
    import torch

    csizes, chost, _ = el.epic_plan_compile(list(wl.chunk_lens), chunk_blocks, n_dummy, cfg.attn, free, num_blocks)
    cplan = el.DevicePlan(csizes, chost, device)
    h = torch.from_numpy(compile_rows(wl, n_dummy)).to(device)
    ws = torch.empty(max(256, el.epic_model_workspace_bytes(cfg, csizes)), dtype=torch.uint8, device=device)
    return CompileStage(cfg=cfg, layers=layers, final_norm=final_norm, sizes=csizes,
                        views=el.plan_views(csizes, chost), dplan=cplan, emb=h, hidden=torch.empty_like(h),
                        out=torch.empty_like(h), workspace=ws)


def stage_model(wl, n_layers: int = None, caches: str = "compile", cache_scale: float = 0.5, device="cuda",
                threads: int = 8, weights_on_device: bool = False, n_dummy: int = 0,
                keep_compile: bool = False, weights: List[Dict[str, object]] = None,
                rerotate: bool = False, tile_rows: int = 0, split_blocks: int = 0) -> ModelStage:
    """Weights, per-chunk caches, link plan and S-row embeddings for a model-level workload.

    caches="compile": every chunk is compiled on the GPU by the library itself
    (epic_plan_compile + epic_link_model, positions 0..L-1; with n_dummy > 0,
    LegoLink-0's compile: n_dummy copies of one dummy token first, dropped after);
    caches="synthetic": every layer's chunk caches are seeded N(0, cache_scale^2) draws;
    caches="none": the pool stays zero (for k < 0, where no cached row is read).
    weights: per-layer device tensors from an earlier stage of the same shape, reused.
    rerotate: the link request re-rotates cached K to its linked positions.
    tile_rows: force the attention tile size of the link plan (0: the planner's choice).
    split_blocks: force the split-KV size of the link plan (0: the planner's choice).
    weights_on_device: draw the weights with a seeded device generator (timing runs)
    instead of synth.model_weights (parity runs).
    """
    import torch

    L = n_layers or wl.n_layers
    cfg = model_cfg(wl, L, tile_rows, split_blocks)
    hq, hkv, d, H = wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.hidden
    acfg = cfg.attn
    given, weights, layers = weights, [], []
    for layer in range(L):
        if given is not None:
            tw = given[layer]
        elif weights_on_device:
            tw = _device_weights(wl, layer, device)
        else:
            w = synth.model_weights(wl.seed, layer, H, wl.ffn, hq, hkv, d, threads=threads)
            tw = {k: _bf16_tensor(v, device) for k, v in w.items()}
        weights.append(tw)
        layers.append(el.epic_layer_weights(*(tw[k].data_ptr() for k in
                                              ("attn_norm", "wqkv", "wo", "mlp_norm", "w_gate_up", "w_down"))))
    final_norm = _bf16_tensor(synth.final_norm_weight(wl.seed, H), device)

    m = len(wl.chunk_lens)
    nb = [-(-x // el.BLOCK) for x in wl.chunk_lens]
    link_req0 = el.Request(list(wl.chunk_lens), [[0] * n for n in nb], wl.suffix_len, wl.k, rerotate)
    n_priv = el.epic_plan_sizes_get([link_req0], acfg, 1 << 30).n_private
    # staging blocks of a dummy-token compile; free again once the compile is done
    n_stage = sum(-(-(n_dummy + x) // el.BLOCK) for x in wl.chunk_lens) if n_dummy > 0 else 0
    num_blocks = sum(nb) + max(n_priv, n_stage, 1)
    perm = np.random.default_rng([wl.seed, 99]).permutation(num_blocks).astype(np.int32)
    chunk_blocks, nxt = [], 0
    for n in nb:
        chunk_blocks.append(perm[nxt:nxt + n].tolist())
        nxt += n
    free = perm[nxt:]
    k_caches = [torch.zeros((num_blocks, hkv, el.BLOCK, d), dtype=torch.bfloat16, device=device) for _ in range(L)]
    v_caches = [torch.zeros((num_blocks, hkv, d, el.BLOCK), dtype=torch.bfloat16, device=device) for _ in range(L)]

    if caches == "compile" and m > 0:
        cst = stage_compile(wl, cfg, layers, final_norm, chunk_blocks, free, num_blocks, n_dummy, device)
        cst.run(k_caches, v_caches)
        torch.cuda.synchronize()
        if not keep_compile:
            cst = None
    elif caches == "synthetic":
        for layer in range(L):
            kp = np.zeros((num_blocks, hkv, el.BLOCK, d), np.uint16)
            vp = np.zeros((num_blocks, hkv, d, el.BLOCK), np.uint16)
            for j, n_tok in enumerate(wl.chunk_lens):
                kr, vr = synth.chunk_cache(wl.seed, j, n_tok, hkv, d, cache_scale, layer=layer)
                kb, vb = el.pack_blocks(kr, vr)
                kp[chunk_blocks[j]] = kb
                vp[chunk_blocks[j]] = vb
            k_caches[layer] = _bf16_tensor(kp, device)
            v_caches[layer] = _bf16_tensor(vp, device)

    req = el.Request(list(wl.chunk_lens), chunk_blocks, wl.suffix_len, wl.k, rerotate)
    sizes, host, views = el.epic_plan_link([req], acfg, free, num_blocks)
    dplan = el.DevicePlan(sizes, host, device)
    emb = _tok_rows(wl, list(range(m)), wl.chunk_lens, wl.suffix_len, views["s_pos"])
    emb_t = torch.from_numpy(emb).to(device)
    ws = torch.empty(max(256, el.epic_model_workspace_bytes(cfg, sizes)), dtype=torch.uint8, device=device)
    return ModelStage(wl=wl, cfg=cfg, weights=weights, layers=layers, final_norm=final_norm, k_caches=k_caches,
                      v_caches=v_caches, requests=[req], chunk_block_ids=chunk_blocks, sizes=sizes, views=views,
                      dplan=dplan, emb=emb_t, hidden=torch.empty_like(emb_t), out=torch.empty_like(emb_t),
                      workspace=ws, compile_stage=cst if caches == "compile" and m > 0 else None)


def gemm_flops_per_layer(wl, n_rows: int) -> float:
    """2 * rows * (sum of in * out over the layer's weight matrices)."""
    qkv = (wl.num_q_heads + 2 * wl.num_kv_heads) * wl.head_dim
    return 2.0 * n_rows * wl.hidden * (qkv + wl.num_q_heads * wl.head_dim + 3 * wl.ffn)


def capture_graph(run):
    """Capture one call of `run` (a staged step that allocates nothing and launches
    only kernels and device copies on the current stream) into a HIP graph; returns
    the torch graph object, whose replay() reruns the step.  One eager call on a side
    stream first, as graph capture expects warmed-up work."""
    import torch

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run()
    torch.cuda.synchronize()
    return graph
