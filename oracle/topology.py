"""UNet topology: the canonical weight table and the conv/linear FLOP count.

Test infrastructure only (see the package docstring).

The configuration object is duck-typed: it carries the fields of the C
``dn_config`` struct (``model_channels``, ``levels`` as a list of
``(channels, depth, heads, head_dim)``, ``layers_per_block``, ``mid_depth``,
``tiny_topology``, ``latent_c``, ``ctx_dim``, ``ff_mult`` ...).

The layout follows the latent-diffusion UNet that the paper's Table 3 sizes
(SD-XL, SD 2.0): a down path of ResNet blocks (with spatial transformers on
levels whose ``depth`` > 0) and stride-2 downsamples, an optional middle block,
and an up path with one more layer per level, each concatenating a skip
activation, with nearest x2 upsample + conv between levels. Parameter counts
are pinned against Table 3 in the tests.

Canonical tensor order (the weight blob is these tensors back to back, fp32,
PyTorch layouts: conv [Cout][Cin][kh][kw], linear [out][in]):
  1. time MLP: lin1.w [4C0, C0], lin1.b, lin2.w [4C0, 4C0], lin2.b
  2. conv_in.w [C0, latent_c, 3, 3], conv_in.b
  3. down levels l = 0..L-1: layers_per_block x (ResBlock, then Transformer if depth_l > 0),
     then (l < L-1) downsample conv [C_l, C_l, 3, 3] + bias
  4. middle (mid_depth >= 0): ResBlock, Transformer(mid_depth) if mid_depth > 0, ResBlock
  5. up levels l = L-1..0: (layers_per_block + 1) x (ResBlock on [h, skip], Transformer if depth_l > 0),
     then (l > 0) upsample conv [C_l, C_l, 3, 3] + bias
  6. out head: gn.g, gn.b [C0], conv_out.w [latent_c, C0, 3, 3], conv_out.b
ResBlock:    gn1.g gn1.b [Cin], conv1.w [Cout, Cin, 3, 3] conv1.b, temb.w [Cout, 4C0] temb.b,
             gn2.g gn2.b [Cout], conv2.w [Cout, Cout, 3, 3] conv2.b, and if Cin != Cout
             skip.w [Cout, Cin, 1, 1] skip.b
Transformer: gn.g gn.b, proj_in.w [C, C] proj_in.b, depth x block, proj_out.w [C, C] proj_out.b
block:       ln1.g ln1.b, attn1.q attn1.k attn1.v [C, C] (no bias), attn1.o.w [C, C] attn1.o.b,
             ln2.g ln2.b, attn2.q [C, C], attn2.k attn2.v [C, ctx_dim], attn2.o.w attn2.o.b,
             ln3.g ln3.b, ff1.w [2 F C, C] ff1.b, ff2.w [C, F C] ff2.b        (F = ff_mult)
The tiny topology is conv_in -> ResBlock -> Transformer(depth_0) -> out head (level 0 only,
no skips, no mid, no up path).

Each table entry is (name, shape, kind, fan_in) with kind in
{"w", "b", "g" (norm scale), "beta" (norm shift)}; fan_in is the layer's input
size (Cin * kh * kw or in_features) and is also given for its bias.
"""

import numpy as np


class _Table:
    def __init__(self):
        self.rows = []

    def w(self, name, shape):
        shape = tuple(int(s) for s in shape)
        fan = int(np.prod(shape[1:]))
        self.rows.append((name + ".w", shape, "w", fan))
        return fan

    def wb(self, name, shape):
        fan = self.w(name, shape)
        self.rows.append((name + ".b", (int(shape[0]),), "b", fan))

    def norm(self, name, c):
        self.rows.append((name + ".g", (int(c),), "g", 0))
        self.rows.append((name + ".b", (int(c),), "beta", 0))


def _res(t, p, cin, cout, temb_dim):
    t.norm(p + ".gn1", cin)
    t.wb(p + ".conv1", (cout, cin, 3, 3))
    t.wb(p + ".temb", (cout, temb_dim))
    t.norm(p + ".gn2", cout)
    t.wb(p + ".conv2", (cout, cout, 3, 3))
    if cin != cout:
        t.wb(p + ".skip", (cout, cin, 1, 1))


def _tx(t, p, c, depth, ctx_dim, ff):
    t.norm(p + ".gn", c)
    t.wb(p + ".proj_in", (c, c))
    for k in range(depth):
        b = f"{p}.blk{k}"
        t.norm(b + ".ln1", c)
        t.w(b + ".attn1.q", (c, c))
        t.w(b + ".attn1.k", (c, c))
        t.w(b + ".attn1.v", (c, c))
        t.wb(b + ".attn1.o", (c, c))
        t.norm(b + ".ln2", c)
        t.w(b + ".attn2.q", (c, c))
        t.w(b + ".attn2.k", (c, ctx_dim))
        t.w(b + ".attn2.v", (c, ctx_dim))
        t.wb(b + ".attn2.o", (c, c))
        t.norm(b + ".ln3", c)
        t.wb(b + ".ff1", (2 * ff * c, c))
        t.wb(b + ".ff2", (c, ff * c))
    t.wb(p + ".proj_out", (c, c))


def walk(cfg):
    """Yield the module sequence of one UNet evaluation as tuples, in forward
    (and canonical-weight) order:
      ("time",), ("conv_in", cout), ("res", prefix, cin, cout), ("tx", prefix, c, depth, heads),
      ("push",), ("down", prefix, c), ("pop_concat",), ("up", prefix, c), ("out", cin)
    Spatial bookkeeping is left to the consumer."""
    c0 = cfg.model_channels
    levels = list(cfg.levels)
    yield ("time",)
    yield ("conv_in", c0)
    if cfg.tiny_topology:
        c, depth, heads, _ = levels[0]
        yield ("res", "down0.0.res", c0, c)
        if depth > 0:
            yield ("tx", "down0.0.tx", c, depth, heads)
        yield ("out", c)
        return
    yield ("push",)
    ch = c0
    L = len(levels)
    for l, (c, depth, heads, _) in enumerate(levels):
        for j in range(cfg.layers_per_block):
            yield ("res", f"down{l}.{j}.res", ch, c)
            ch = c
            if depth > 0:
                yield ("tx", f"down{l}.{j}.tx", c, depth, heads)
            yield ("push",)
        if l < L - 1:
            yield ("down", f"down{l}.down", c)
            yield ("push",)
    if cfg.mid_depth >= 0:
        c, _, heads, _ = levels[-1]
        yield ("res", "mid.res0", ch, c)
        if cfg.mid_depth > 0:
            yield ("tx", "mid.tx", c, cfg.mid_depth, heads)
        yield ("res", "mid.res1", c, c)
    for l in reversed(range(L)):
        c, depth, heads, _ = levels[l]
        for j in range(cfg.layers_per_block + 1):
            yield ("pop_concat",)
            yield ("res", f"up{l}.{j}.res", None, c)   # Cin = ch + skip channels, known at run time
            ch = c
            if depth > 0:
                yield ("tx", f"up{l}.{j}.tx", c, depth, heads)
        if l > 0:
            yield ("up", f"up{l}.up", c)
    yield ("out", ch)


def _skip_channels(cfg):
    """Channels of each pushed skip activation, in push order."""
    c0 = cfg.model_channels
    out = [c0]
    levels = list(cfg.levels)
    for l, (c, _, _, _) in enumerate(levels):
        out += [c] * cfg.layers_per_block
        if l < len(levels) - 1:
            out.append(c)
    return out


def tensor_table(cfg):
    """Canonical weight table [(name, shape, kind, fan_in)] for a configuration."""
    c0 = cfg.model_channels
    temb = 4 * c0
    t = _Table()
    skips = [] if cfg.tiny_topology else _skip_channels(cfg)
    ch = c0
    for op in walk(cfg):
        kind = op[0]
        if kind == "time":
            t.wb("time.lin1", (temb, c0))
            t.wb("time.lin2", (temb, temb))
        elif kind == "conv_in":
            t.wb("conv_in", (c0, cfg.latent_c, 3, 3))
        elif kind == "pop_concat":
            ch = ch + skips.pop()
        elif kind == "res":
            _, p, _, cout = op
            _res(t, p, ch, cout, temb)
            ch = cout
        elif kind == "tx":
            _, p, c, depth, _ = op
            _tx(t, p, c, depth, cfg.ctx_dim, cfg.ff_mult)
        elif kind in ("down", "up"):
            _, p, c = op
            t.wb(p, (c, c, 3, 3))
        elif kind == "out":
            t.norm("out.gn", op[1])
            t.wb("conv_out", (cfg.latent_c, op[1], 3, 3))
    return t.rows


def param_count(cfg):
    return int(sum(int(np.prod(s)) for _, s, _, _ in tensor_table(cfg)))


def flop_count(cfg, n, h, w):
    """FLOPs of one UNet evaluation on n samples at latent size h x w, at 2 FLOP per
    multiply-add. Returns (conv_linear, attention_matmuls): the first counts every
    conv and linear layer (the quantity Table 3 reports), the second the two
    batched products of each attention (Q K^T and P V)."""
    c0 = cfg.model_channels
    temb = 4 * c0
    lin = 0.0
    att = 0.0
    ch = c0
    hh, ww = h, w
    skips = [] if cfg.tiny_topology else _skip_channels(cfg)
    for op in walk(cfg):
        kind = op[0]
        if kind == "time":
            lin += 2 * n * (c0 * temb + temb * temb)
        elif kind == "conv_in":
            lin += 2 * n * hh * ww * c0 * cfg.latent_c * 9
        elif kind == "pop_concat":
            ch = ch + skips.pop()
        elif kind == "res":
            cout = op[3]
            px = n * hh * ww
            lin += 2 * px * cout * ch * 9 + 2 * px * cout * cout * 9 + 2 * n * temb * cout
            if ch != cout:
                lin += 2 * px * cout * ch
            ch = cout
        elif kind == "tx":
            _, _, c, depth, _ = op
            s = hh * ww
            tok = n * s
            lin += 2 * 2 * tok * c * c  # proj_in, proj_out
            per = (2 * tok * c * c * 4             # q k v o (self)
                   + 2 * tok * c * c * 2           # q, o (cross)
                   + 2 * n * cfg.ctx_len * cfg.ctx_dim * c * 2  # k, v of the context
                   + 2 * tok * c * 2 * cfg.ff_mult * c          # ff1
                   + 2 * tok * cfg.ff_mult * c * c)             # ff2
            lin += depth * per
            att += depth * (2 * 2 * n * s * s * c + 2 * 2 * n * s * cfg.ctx_len * c)
        elif kind == "down":
            c = op[2]
            hh, ww = hh // 2, ww // 2
            lin += 2 * n * hh * ww * c * c * 9
        elif kind == "up":
            c = op[2]
            hh, ww = hh * 2, ww * 2
            lin += 2 * n * hh * ww * c * c * 9
        elif kind == "out":
            lin += 2 * n * hh * ww * cfg.latent_c * op[1] * 9
    return lin, att
