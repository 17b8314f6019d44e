"""Helpers for the GPU parity tests and the benchmark (no method arithmetic)."""
import numpy as np
import torch


def to_oracle(x: torch.Tensor) -> np.ndarray:
    """A logits tensor as the oracle takes it: fp32 array, or bf16 bit patterns as uint16."""
    x = x.detach().cpu()
    if x.dtype == torch.float32:
        return x.numpy()
    if x.dtype == torch.bfloat16:
        return x.view(torch.int16).numpy().view(np.uint16)
    raise TypeError(x.dtype)


def u32(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy().view(np.uint32)


def run_chain(dv, ns, al, init_states: torch.Tensor, logits_all: torch.Tensor, ws):
    """Greedy chain on the device, as the benchmark runs it: step k reads
    states_all[k] and writes states_all[k + 1] and tokens_all[k]."""
    steps, B = logits_all.shape[0], logits_all.shape[1]
    dev = init_states.device
    states_all = torch.empty((steps + 1, B), dtype=torch.int32, device=dev)
    tokens_all = torch.empty((steps, B), dtype=torch.int32, device=dev)
    states_all[0].copy_(init_states)
    for k in range(steps):
        dv.masked_step(ns, al, states_all[k], logits_all[k], token=tokens_all[k],
                       new_state=states_all[k + 1], workspace=ws)
    return tokens_all, states_all
