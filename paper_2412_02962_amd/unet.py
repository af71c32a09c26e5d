"""One band's SDXL-shaped U-Net forward on the GPU, composed of the
library's C-ABI calls: pcpp_conv3x3 (conv_in, the down- and upsamplers,
conv_out), pcpp_resnet_block, pcpp_transformer_module (the partially
conditioned self-attention of Sec. 3.3 inside), pcpp_concat_channels (the up
path's skip connections) and pcpp_group_norm (the output head).  This module
only plans buffers and marshals arguments; every step runs in the library's
kernels.

The layer order and shapes come from synth.unet_layers; the weights and the
band's stale neighbour data of the previous step (the rows above and below
each convolution input, the ResNets' edge rows, every basic block's K/V) are
inputs, as the neighbour exchange (Sec. 3.2) delivers them.  GroupNorms use
the band's own statistics, or with sync_gn every band's (Sec. 3.3).
"""

from __future__ import annotations

from typing import Dict, List

from . import pcpp


class BandUNet:
    def __init__(self, sp, layers: List[dict], weights: Dict, stale: Dict, device="cuda:0", sync_gn=False):
        """sync_gn: every GroupNorm uses the whole image's statistics (Sec. 3.3),
        from every band's (count, mean, M2) in stale (resnet: gn1_bands and
        gn2_bands; module NAME: stale[NAME + ':gn_bands']; output head:
        gn_bands); the band's own statistics are written to self.gn_own."""
        import torch
        self.sp, self.layers = sp, layers
        self.weights, self.stale = weights, stale
        self.sync_gn = sync_gn
        self.gn_own = {}
        B, n, i = sp.batch, sp.n, sp.i
        self.plans = []
        ws_max = 0
        for ly in layers:
            H, W, ci, co = ly["H"], ly["W"], ly["c_in"], ly["c_out"]
            h = H // n
            plan = {"ly": ly}
            w = weights[ly["name"]]
            if ly["kind"] == "conv":
                g = pcpp.make_conv_geom(H, W, n, i, ci, co, B, ly["mode"])
                tok = {0: h * W, 1: (h // 2) * (W // 2), 2: 4 * h * W}[ly["mode"]]
                plan.update(g=g, out=torch.empty((B, tok, co), dtype=torch.bfloat16, device=device))
                wsb = pcpp.pcpp_conv3x3_workspace_size(g)
            elif ly["kind"] == "resnet":
                g = pcpp.make_resnet_geom(H, W, n, i, ci, co, sp.temb_dim, sp.groups, B, 1e-5)
                plan.update(g=g, wts=pcpp.make_resnet_weights(w),
                            out=torch.empty((B, h * W, co), dtype=torch.bfloat16, device=device))
                if ly.get("pop"):
                    plan["cat"] = torch.empty((B, h * W, ci), dtype=torch.bfloat16, device=device)
                wsb = pcpp.pcpp_resnet_block_workspace_size(g)
            elif ly["kind"] == "module":
                g = pcpp.make_geom(H, W, n, i, sp.p, w["heads"], 64, B, 0, pcpp.PCPP_DTYPE_BF16)
                # p = 0: the band's attention without stale rows (a band computed on its own)
                g0 = pcpp.make_geom(H, W, n, i, 0.0, w["heads"], 64, B, 0, pcpp.PCPP_DTYPE_BF16)
                mw, keep = pcpp.make_module_weights(w["module"], w["blocks"], w["ff_inner"], sp.groups)
                plan.update(g=g, g0=g0, wts=mw, keep=keep,
                            out=torch.empty((B, h * W, co), dtype=torch.bfloat16, device=device))
                wsb = pcpp.pcpp_transformer_module_workspace_size(g, mw, sp.n_text, sp.text_dim)
            else:
                plan.update(out=torch.empty((B, h * W, co), dtype=torch.bfloat16, device=device))
                wsb = pcpp.pcpp_group_norm_workspace_size(B, h * W, co, sp.groups)
            if wsb == 0:
                raise ValueError(f"layer {ly['name']}: the library rejects its shape")
            if sync_gn:
                own = lambda: torch.empty((B, sp.groups, 3), dtype=torch.float32, device=device)
                self.gn_own[ly["name"]] = [own(), own()] if ly["kind"] == "resnet" else (
                    [own()] if ly["kind"] in ("module", "gn") else [])
            ws_max = max(ws_max, wsb)
            self.plans.append(plan)
        # One workspace for all layers: every call treats it as scratch (the
        # module clears the work counters its launches use).
        self.ws = torch.empty(ws_max, dtype=torch.uint8, device=device)
        self.ws_bytes = ws_max

    def forward(self, latent, temb, text, stale=None, exports=None, gn_own=None, separate=False):
        """latent [B, h*W0, 64] (4 channels, zero-padded), temb [B, T], text
        [B, n_text, text_dim] (device bf16) -> the band's noise prediction
        [B, h*W0, 64] (channels 4.. are zero; the buffer is reused by the
        next call).  stale replaces the constructor's stale data for this
        call.  exports (per layer, optional) receives what the neighbours
        read at the next step: a convolution's first / last input rows
        ('first', 'last' [B, W, c_in]), a ResNet's 'edges1' / 'edges2', a
        module's per-block 'k' / 'v' lists.  gn_own replaces self.gn_own (the
        band's own GroupNorm statistics, per layer a list).  separate: the
        attention layers take no stale rows (p = 0), as for a band computed
        on its own before anything has been exchanged; the modules' stale
        K/V are then not read."""
        sp, ws, wsb = self.sp, self.ws, self.ws_bytes
        B = sp.batch
        stale = self.stale if stale is None else stale
        own_all = self.gn_own if gn_own is None else gn_own
        cur = latent
        skips = []
        for plan in self.plans:
            ly = plan["ly"]
            name, out = ly["name"], plan["out"]
            w = self.weights[name]
            ex = exports.get(name) if exports is not None else None
            if ly["kind"] == "conv":
                st = stale[name]
                if ex is not None:
                    pcpp.pcpp_conv3x3_export(plan["g"], cur, st["row_up"], st["row_dn"], w["w"], w["b"], out,
                                             ex["first"], ex["last"], ws, wsb)
                else:
                    pcpp.pcpp_conv3x3(plan["g"], cur, st["row_up"], st["row_dn"], w["w"], w["b"], out, ws, wsb)
            elif ly["kind"] == "resnet":
                if ly.get("pop"):
                    skip = skips.pop()
                    rows = cur.shape[0] * cur.shape[1]
                    pcpp.pcpp_concat_channels(rows, cur, cur.shape[2], skip, skip.shape[2], plan["cat"])
                    cur = plan["cat"]
                st = stale[name]
                b1, b2 = (st["gn1_bands"], st["gn2_bands"]) if self.sync_gn else (None, None)
                o1, o2 = own_all[name] if self.sync_gn else (None, None)
                e1, e2 = (ex["edges1"], ex["edges2"]) if ex is not None else (None, None)
                pcpp.pcpp_resnet_block(plan["g"], plan["wts"], cur, temb, st["edges1_up"], st["edges1_dn"],
                                       st["edges2_up"], st["edges2_dn"], b1, o1, b2, o2, out, e1, e2, ws, wsb)
            elif ly["kind"] == "module":
                if separate:
                    ku = vu = kd = vd = None
                else:
                    cols = list(zip(*stale[name]))
                    ku, vu, kd, vd = [None if any(a is None for a in c) else list(c) for c in cols]
                bands = stale[name + ":gn_bands"] if self.sync_gn else None
                own = own_all[name][0] if self.sync_gn else None
                ko, vo = (ex["k"], ex["v"]) if ex is not None else (None, None)
                pcpp.pcpp_transformer_module(plan["g0"] if separate else plan["g"], plan["wts"], cur, text, sp.n_text, sp.text_dim, ku, vu, kd,
                                             vd, bands, own, out, ko, vo, ws, wsb)
            else:
                bands = stale[name]["gn_bands"] if self.sync_gn else None
                own = own_all[name][0] if self.sync_gn else None
                pcpp.pcpp_group_norm(B, cur.shape[1], cur.shape[2], sp.groups, 1e-5, 1, cur, w["gamma"], w["beta"],
                                     out, ws, wsb, bands=bands, n_bands=sp.n, band=sp.i, own_out=own)
            if ly.get("push"):
                skips.append(out)
            cur = out
        return cur
