"""A torch-library formulation of the expert (test-only), used to pin the oracle.

The recurrent body is ``torch.nn.LSTM(bias=False)`` (gate order i, f, g, o),
the embedding a row gather, the head a bias-free linear map and the loss
``F.cross_entropy``: library routines, not a retyping of the oracle.  The flat
parameter vector uses the canonical layout Emb[V][E]; W_l[4H][in_l + H]
(columns [input | recurrent]); Whead[V][H].
"""
import torch
import torch.nn.functional as F
from torch.func import functional_call

V = 256


def split(theta: torch.Tensor, n_layers: int, embed: int, hidden: int):
    off = 0
    emb = theta[off: off + V * embed].reshape(V, embed)
    off += V * embed
    params = {}
    for l in range(n_layers):
        ind = embed if l == 0 else hidden
        W = theta[off: off + 4 * hidden * (ind + hidden)].reshape(4 * hidden, ind + hidden)
        off += 4 * hidden * (ind + hidden)
        params[f"weight_ih_l{l}"] = W[:, :ind]
        params[f"weight_hh_l{l}"] = W[:, ind:]
    head = theta[off: off + V * hidden].reshape(V, hidden)
    assert off + V * hidden == theta.numel()
    return emb, params, head


def loss(theta: torch.Tensor, n_layers: int, embed: int, hidden: int, bytes_e) -> torch.Tensor:
    """Mean next-byte cross entropy of one expert on its batch [B][T]."""
    x = torch.as_tensor(bytes_e, dtype=torch.long)
    emb, params, head = split(theta, n_layers, embed, hidden)
    lstm = torch.nn.LSTM(embed, hidden, num_layers=n_layers, bias=False, batch_first=True)
    lstm = lstm.to(theta.dtype)
    out, _ = functional_call(lstm, params, (emb[x[:, :-1]],))
    logits = out @ head.T
    return F.cross_entropy(logits.reshape(-1, V), x[:, 1:].reshape(-1))
