"""Helpers of the GPU parity tests: device transfer of the seeded inputs and
the comparison rules (tolerances are stated where they are used)."""
import numpy as np
import torch

import synth


def dev_bf16(bits):
    a = np.ascontiguousarray(bits).view(np.int16)
    return torch.from_numpy(a).view(torch.bfloat16).cuda()


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def f32(bits):
    return synth.bf16_bits_to_f32(bits)


def host_bf16_f32(t):
    return synth.bf16_bits_to_f32(t.detach().view(torch.int16).cpu().numpy().view(np.uint16))
