"""One denoising step of the whole image under PCPP on one device: every
band's U-Net forward (BandUNet, all of it C-ABI calls), band after band,
each with the stale data its neighbours exported at the previous step
(Sec. 3.2: the exchange that devices do over the network).  Here the
exchange costs nothing: each band's exports are written by the library's
kernels straight into buffers that the neighbours read one step later
(two sets, by step parity, so a band never overwrites what another band
of the same step still reads).  This module only allocates buffers and
hands pointers around.

What band i reads from band i-1 (from band i+1 the mirror image):
  convolution     its last input row (row_up; the first one is row_dn)
  ResNet          its edge rows [B, 2, W, C] (the kernel reads the last)
  self-attention  every basic block's K and V (the attention reads the
                  last r rows)
  GroupNorm       with synchronized statistics, every band's (count, mean,
                  M2) of the step before, stacked [n, B, G, 3]
Before the first step nothing has been received, and with no synchronous
warm-up step the bands are computed separately (as in the paper's Fig. 1):
the attention layers take no stale rows (p = 0 for that step), the
convolutions read zero rows beyond the band and the GroupNorm statistics of
the other bands have count 0 (the merge skips them).
"""

from __future__ import annotations

import dataclasses
from typing import Dict, List

from .unet import BandUNet


class ImageStep:
    def __init__(self, sp, layers: List[dict], weights: Dict, device="cuda:0", sync_gn=True):
        import torch
        self.sp, self.layers, self.sync_gn = sp, layers, sync_gn
        n, B, G = sp.n, sp.batch, sp.groups
        bf = torch.bfloat16
        zeros = lambda *shape: torch.zeros(shape, dtype=bf, device=device)
        self.nets = [BandUNet(dataclasses.replace(sp, i=i), layers, weights, None, device, sync_gn)
                     for i in range(n)]

        def band_exports():
            ex = {}
            for ly in layers:
                W, ci, co, h = ly["W"], ly["c_in"], ly["c_out"], ly["H"] // n
                if ly["kind"] == "conv":
                    ex[ly["name"]] = {"first": zeros(B, W, ci), "last": zeros(B, W, ci)}
                elif ly["kind"] == "resnet":
                    ex[ly["name"]] = {"edges1": zeros(B, 2, W, ci), "edges2": zeros(B, 2, W, co)}
                elif ly["kind"] == "module":
                    ex[ly["name"]] = {"k": [zeros(B, h * W, co) for _ in range(ly["depth"])],
                                      "v": [zeros(B, h * W, co) for _ in range(ly["depth"])]}
            return ex

        def gn_stacks():  # per layer, one [n, B, G, 3] stack per GroupNorm of the layer
            sites = {"resnet": 2, "module": 1, "gn": 1}
            return {ly["name"]: [torch.zeros((n, B, G, 3), dtype=torch.float32, device=device)
                                 for _ in range(sites.get(ly["kind"], 0))] for ly in layers}

        self.exports = [[band_exports() for _ in range(n)] for _ in range(2)]
        self.stats = [gn_stacks() for _ in range(2)] if sync_gn else None
        self.t = 0

    def _stale(self, i, prev):
        """Band i's stale data from the neighbours' exports in set `prev`."""
        n = self.sp.n
        up = self.exports[prev][i - 1] if i > 0 else None
        dn = self.exports[prev][i + 1] if i < n - 1 else None
        st = {}
        for ly in self.layers:
            name, kind = ly["name"], ly["kind"]
            if kind == "conv":
                st[name] = {"row_up": up[name]["last"] if up else None,
                            "row_dn": dn[name]["first"] if dn and ly["mode"] != 1 else None}
            elif kind == "resnet":
                st[name] = {"edges1_up": up[name]["edges1"] if up else None,
                            "edges1_dn": dn[name]["edges1"] if dn else None,
                            "edges2_up": up[name]["edges2"] if up else None,
                            "edges2_dn": dn[name]["edges2"] if dn else None}
                if self.sync_gn:
                    st[name]["gn1_bands"], st[name]["gn2_bands"] = self.stats[prev][name]
            elif kind == "module":
                st[name] = [(up[name]["k"][j] if up else None, up[name]["v"][j] if up else None,
                             dn[name]["k"][j] if dn else None, dn[name]["v"][j] if dn else None)
                            for j in range(ly["depth"])]
                if self.sync_gn:
                    st[name + ":gn_bands"] = self.stats[prev][name][0]
            else:
                st[name] = {"gn_bands": self.stats[prev][name][0] if self.sync_gn else None}
        return st

    def step(self, latents, temb, text):
        """latents[i]: band i's [B, h*W0, 64] input; returns the bands' noise
        predictions (buffers reused by the next step)."""
        cur, prev = self.t % 2, (self.t + 1) % 2
        outs = []
        for i, net in enumerate(self.nets):
            own = ({name: [s[i] for s in stacks] for name, stacks in self.stats[cur].items()}
                   if self.sync_gn else None)
            outs.append(net.forward(latents[i], temb, text, stale=self._stale(i, prev),
                                    exports=self.exports[cur][i], gn_own=own, separate=self.t == 0))
        self.t += 1
        return outs
