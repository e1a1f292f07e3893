"""A hybrid layer stack for the end-to-end GPU tests (test code).

The stack owns the live buffer set of a hybrid model -- per linear layer a
recurrent state [H, dk, dv] fp32 and a conv tail [W, C] bf16, per
full-attention layer positional K and V buffers [T_max, kv_heads, d] bf16 --
and drives it through the library: every linear layer's prefill or decode
step is a linattn_chunked_prefill call (mixer "linattn") or a
gdn_chunked_prefill call (mixer "gdn", the gated delta rule) that reads and
writes the layer's live state in place; snapshot / restore / fork go through
the capsule calls.

What the out-of-scope parts of a model would produce is replaced by seeded
synthetic tables (synth): the per-token q/k/v/g of each linear layer, the K/V
rows each full-attention layer appends, and the conv inputs whose last W rows
form the tail.  Those rows enter the live set through the library's append
(cap_set_append: positional K/V rows, sliding conv windows).
"""
import numpy as np
import torch

import paper_2606_20537_amd as cap
import synth


class HybridStack:
    def __init__(self, w, total_tokens, stream_seed=0, inputs=None, deploy_key=0x5EED, mixer="linattn"):
        self.w = w
        self.mixer = mixer
        self.T_total = total_tokens
        assert total_tokens <= w.t_max
        dev = torch.device("cuda")
        self.dev = dev
        H, dk, dv = w.heads, w.dk, w.dv
        seed = w.seed + 1000 * stream_seed
        # per-layer synthetic inputs over [0, total_tokens)
        if inputs is None:
            inputs = make_inputs(w, total_tokens, seed, mixer)
        self.inp = inputs
        self.ws = None
        if mixer == "gdn":  # scratch of the delta-rule prefill, sized for the longest call
            self.ws = torch.empty(max(cap.gdn_workspace_bytes(total_tokens, H), 16), dtype=torch.uint8, device=dev)
        # live buffers
        self.state = [torch.zeros((H, dk, dv), dtype=torch.float32, device=dev) for _ in range(w.n_linear)]
        cw, cc = w.conv_width, w.conv_channels
        self.conv = [torch.zeros((max(cw, 1), max(cc, 8)), dtype=torch.bfloat16, device=dev) for _ in range(w.n_linear)]
        self.kv = [torch.zeros((w.t_max, w.kv_heads, w.kv_dim), dtype=torch.bfloat16, device=dev)
                   for _ in range(2 * w.n_full)]
        self.o = [torch.full((total_tokens, H, dv), float("nan"), dtype=torch.float32, device=dev)
                  for _ in range(w.n_linear)]
        bufs = []
        li = ki = 0
        for layer in range(w.n_linear + w.n_full):
            if (layer % 4 == 3 and ki < len(self.kv)) or li >= w.n_linear:
                for _ in range(2):
                    t = self.kv[ki]
                    bufs.append(("kv%d" % ki, t, w.kv_row_bytes, w.t_max, cap.CAP_KIND_POSITIONAL))
                    ki += 1
            else:
                bufs.append(("state%d" % li, self.state[li], H * dk * dv * 4, 1, cap.CAP_KIND_FIXED))
                c = self.conv[li]  # a window of W rows of C bf16
                bufs.append(("conv%d" % li, c, c.shape[1] * 2, c.shape[0], cap.CAP_KIND_FIXED))
                li += 1
        self.bufs = bufs
        self.set = cap.cap_set_create(bufs, w.chunk, deploy_key)
        self.pos = 0

    # --- the model's other layers, replaced by synthetic tables -----------
    def _append_rows(self, t0, t1):
        """The K/V rows and conv inputs of tokens [t0, t1) enter the set
        (one cap_set_append launch; the states are the scan's)."""
        srcs, ki, li = [], 0, 0
        for name, t, rb, rows, kind in self.bufs:
            if name.startswith("kv"):
                srcs.append(self.inp["kv"][ki][t0:t1])
                ki += 1
            elif name.startswith("conv"):
                srcs.append(self.inp["conv"][li][t0:t1] if self.w.conv_width else None)
                li += 1
            else:
                srcs.append(None)
        cap.cap_set_append(self.set, srcs, t1 - t0)

    # --- the hot path -----------------------------------------------------
    def prefill(self, t0, t1, decode=False):
        """Run tokens [t0, t1) through every linear layer (one call each):
        the chunked prefill, or with decode=True (one token) the decode step."""
        assert t0 == self.pos, (t0, self.pos)
        assert not decode or t1 == t0 + 1
        w = self.w
        T = t1 - t0
        for l in range(w.n_linear):
            d = self.inp["lin"][l]
            if self.mixer == "gdn":
                if decode:
                    cap.gdn_decode_step(d["q"][t0:t1], d["k"][t0:t1], d["v"][t0:t1], d["g"][t0:t1],
                                        d["beta"][t0:t1], self.o[l][t0:t1], state_in=self.state[l],
                                        final_state=self.state[l], T=T, H=w.heads, dk=w.dk, dv=w.dv, chunk=w.chunk)
                else:
                    cap.gdn_chunked_prefill(d["q"][t0:t1], d["k"][t0:t1], d["v"][t0:t1], d["g"][t0:t1],
                                            d["beta"][t0:t1], self.o[l][t0:t1], state_in=self.state[l],
                                            final_state=self.state[l], workspace=self.ws,
                                            T=T, H=w.heads, dk=w.dk, dv=w.dv, chunk=w.chunk)
                continue
            fn = cap.linattn_decode_step if decode else cap.linattn_chunked_prefill
            fn(d["q"][t0:t1], d["k"][t0:t1], d["v"][t0:t1], d["g"][t0:t1],
               self.o[l][t0:t1], state_in=self.state[l], final_state=self.state[l],
               T=T, H=w.heads, dk=w.dk, dv=w.dv, chunk=w.chunk,
               in_dtype=cap.CAP_DTYPE_F32 if w.in_dtype == "f32" else cap.CAP_DTYPE_BF16)
        cap.cap_set_set_position(self.set, t0)
        self._append_rows(t0, t1)
        self.pos = t1

    def decode(self, n):
        """n decode steps (one token each, the decode entry points)."""
        for _ in range(n):
            self.prefill(self.pos, self.pos + 1, decode=True)

    def snapshot(self, P, digest=0):
        nbytes = cap.capsule_bytes(self.set, P)
        arena = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=self.dev)
        return cap.capsule_snapshot(self.set, P, digest, arena)

    def restore(self, c, digest=0):
        self.pos = cap.capsule_restore(c, self.set, digest)
        return self.pos

    def poison(self):
        """Overwrite every live byte (adversarial dirtied-state check)."""
        for _, t, _, _, _ in self.bufs:
            t.view(torch.uint8).fill_(0xFF)
        for o in self.o:
            o.fill_(float("nan"))

    def live_bytes(self):
        return [t.view(torch.uint8).clone() for _, t, _, _, _ in self.bufs]


def make_inputs(w, total_tokens, seed, mixer="linattn"):
    dev = torch.device("cuda")
    lin = []
    for l in range(w.n_linear):
        if mixer == "gdn":
            d = synth.gdn_inputs(seed, l, total_tokens, w.heads, w.dk, w.dv, w.in_dtype)
        else:
            d = synth.linattn_inputs(seed, l, total_tokens, w.heads, w.dk, w.dv, w.in_dtype)
        entry = {"host": d}
        for n in ("q", "k", "v"):
            pay = d[n + "_dev"]
            t = torch.from_numpy(pay.view(np.int16).copy()).view(torch.bfloat16) if pay.dtype == np.uint16 \
                else torch.from_numpy(np.ascontiguousarray(pay))
            entry[n] = t.to(dev)
        entry["g"] = torch.from_numpy(d["g"]).to(dev)
        if "beta" in d:
            entry["beta"] = torch.from_numpy(d["beta"]).to(dev)
        lin.append(entry)
    kv = []
    for i in range(2 * w.n_full):
        vals, bits = synth.normal_tensor(seed, 100 + i, "kvrows", (total_tokens, w.kv_heads, w.kv_dim), "bf16")
        kv.append(torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(dev))
    conv = []
    for l in range(w.n_linear if w.conv_width else 0):
        vals, bits = synth.normal_tensor(seed, 200 + l, "convin", (total_tokens, w.conv_channels), "bf16")
        conv.append(torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(dev))
    return {"lin": lin, "kv": kv, "conv": conv}
