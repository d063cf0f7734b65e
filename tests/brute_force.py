"""Independent second formulation of the model, used only to pin the oracle.

Dense incidence matrices replace every index operation: with one-hot
S_src, S_dst in {0,1}^{E x N}, gathering is S @ H and sum aggregation is
S^T @ E'. Linear, LayerNorm, ReLU and sigmoid are torch-CPU library routines
in float64. The weight blob is read through the generator module's named
views, not through the oracle's own parser. Only for tiny graphs.
"""
from __future__ import annotations

import numpy as np
import torch
import torch.nn.functional as Fn

from paper_2402_09633_amd.inputs import blob_views


def incidence(idx: np.ndarray, n_nodes: int) -> torch.Tensor:
    S = torch.zeros(idx.size, n_nodes, dtype=torch.float64)
    if idx.size:
        S[torch.arange(idx.size), torch.as_tensor(idx, dtype=torch.long)] = 1.0
    return S


def forward(blob, x, edge_index, F, H, T, S=1, eps=1e-5):
    V = {k: torch.as_tensor(np.asarray(v, np.float64)) for k, v in
         blob_views(np.asarray(blob, np.float32), F, H, S).items()}
    N = x.shape[0]
    src, dst = np.asarray(edge_index[0]), np.asarray(edge_index[1])
    Ss, Sd = incidence(src, N), incidence(dst, N)

    def hid(name, a):
        y = Fn.linear(a, V[name + ".W"], V[name + ".b"])
        y = Fn.layer_norm(y, (y.shape[-1],), V[name + ".g"], V[name + ".beta"], eps)
        return torch.relu(y)

    def mlp(name, a):
        return hid(name + ".1", hid(name + ".0", a))

    h = mlp("node_enc", torch.as_tensor(np.asarray(x, np.float64)))
    e = mlp("edge_enc", torch.cat([Ss @ h, Sd @ h], 1))
    dumps = [{"h": h, "e": e}]
    for t in range(T):
        k = 0 if S == 1 else t
        e2 = mlp(f"edge_mlp{k}", torch.cat([Ss @ h, Sd @ h, e], 1))
        ain, aout = Sd.T @ e2, Ss.T @ e2
        h2 = mlp(f"node_mlp{k}", torch.cat([h, ain, aout], 1))
        h, e = h2, e2
        dumps.append({"h": h, "e": e, "agg_in": ain, "agg_out": aout})
    c = hid("edge_cls.0", torch.cat([Ss @ h, Sd @ h, e], 1))
    z = Fn.linear(c, V["edge_cls.1.W"], V["edge_cls.1.b"])[:, 0]
    return {"logits": z.numpy(), "scores": torch.sigmoid(z).numpy(),
            "dumps": [{k: v.numpy() for k, v in d.items()} for d in dumps]}
