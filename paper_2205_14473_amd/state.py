"""Device buffers of one round (optimizer state and messages), sized by libea.

Plumbing only: torch allocates; sizes come from the C ABI's size queries.
"""
from dataclasses import dataclass
from typing import Optional

from . import _binding as B


@dataclass
class RoundBuffers:
    g: "object"                 # [N, d] gradients (caller fills)
    e_w: "object"               # [N, d]
    e_s: "object"               # [d]
    x: "object"                 # [d]
    wcodes: "object"            # [N, words_w] uint64
    wscales: "object"           # [N, scales_w]
    scodes: "object"            # [words_s] uint64
    sscales: "object"           # [scales_s]
    m: Optional[object] = None  # [d]    (Adam at the server)
    v: Optional[object] = None
    m_w: Optional[object] = None  # [N, d] (Adam at the workers)
    v_w: Optional[object] = None
    workspace: Optional[object] = None
    u: Optional[object] = None    # [d] split-call intermediate

    def step_args(self):
        return dict(g=self.g, e_w=self.e_w, m_w=self.m_w, v_w=self.v_w, m=self.m, v=self.v, e_s=self.e_s,
                    x=self.x, wcodes=self.wcodes, wscales=self.wscales, scodes=self.scodes,
                    sscales=self.sscales, workspace=self.workspace)


def allocate(cfg: B.Config, device="cuda", with_u: bool = False) -> RoundBuffers:
    import torch
    d, N = cfg.d, cfg.N
    f32 = dict(dtype=torch.float32, device=device)
    ww, sw = B.ea_msg_words(cfg.qw, d), B.ea_msg_words(cfg.qs, d)
    ns_w, ns_s = B.ea_msg_scales(cfg.qw, d), B.ea_msg_scales(cfg.qs, d)
    ws = B.ea_workspace_bytes(cfg)
    rb = RoundBuffers(
        g=torch.empty((N, d), **f32), e_w=torch.empty((N, d), **f32), e_s=torch.empty(d, **f32),
        x=torch.zeros(d, **f32),
        wcodes=torch.zeros((N, ww), dtype=torch.uint64, device=device),
        wscales=torch.zeros((N, max(ns_w, 1)), **f32),
        scodes=torch.zeros(sw, dtype=torch.uint64, device=device),
        sscales=torch.zeros(max(ns_s, 1), **f32),
        workspace=torch.empty(ws, dtype=torch.uint8, device=device) if ws > 0 else None,
        u=torch.empty(d, **f32) if with_u else None,
    )
    if cfg.placement == B.EA_ADAM_AT_WORKER:
        rb.m_w = torch.empty((N, d), **f32)
        rb.v_w = torch.empty((N, d), **f32)
    else:
        rb.m = torch.empty(d, **f32)
        rb.v = torch.empty(d, **f32)
    return rb


def init_state(cfg: B.Config, rb: RoundBuffers, stream=None):
    B.ea_state_init(cfg, rb.m, rb.v, rb.e_s, rb.e_w, rb.m_w, rb.v_w, stream)
