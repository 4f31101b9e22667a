"""Running the HIP path on a generated workload (GPU tests, smoke and bench share this shape)."""
from __future__ import annotations

import numpy as np

from paper_2609_38795_amd import binding, workloads as W


def make_engine(inp, max_anchors=None, max_block=None):
    import torch

    w = inp.workload
    lim = binding.make_limits(w.n_tokens, w.n_seq, max_anchors or w.n_anchors,
                              max_block or w.block)
    return binding.Engine(w.shape, inp.weights, w.max_pos, lim, device=torch.device("cuda:0"))


def prefill(eng, inp, feats=False):
    import torch

    w = inp.workload
    dev = eng.device
    toks = torch.from_numpy(inp.tokens.reshape(-1).astype(np.int32)).to(dev)
    emb = mask = None
    if inp.embeds is not None:
        e = inp.embeds
        emb = torch.from_numpy(e.view(np.int16) if e.dtype == np.uint16 else e).to(dev)
        mask = torch.from_numpy(inp.embed_mask).to(dev)
    fo = None
    if feats and w.shape.n_feat:
        fo = torch.empty((w.n_tokens, w.shape.n_feat, w.shape.d_model), dtype=torch.float32,
                         device=dev)
    eng.prefill(toks, [w.seq_len] * w.n_seq, emb, mask, fo)
    return fo


def runner(eng, a_seq, a_pos, block):
    """gpu_run(forced) -> numpy (tokens, logprobs, feats) for the given anchors."""
    import torch

    def run(forced):
        f = None if forced is None else torch.from_numpy(np.ascontiguousarray(forced, np.int32)).to(eng.device)
        tok, lp, ft = eng.rollout(a_seq, a_pos, block, forced=f)
        torch.cuda.synchronize()
        ftn = ft.cpu().numpy() if ft is not None else np.zeros((len(a_seq), block, 0, 0))
        return tok.cpu().numpy().astype(np.int64), lp.cpu().numpy(), ftn

    return run
