"""Frame-by-frame block-sparse ResNet backbones and SwiftNet-style segmentation
networks with persistent per-layer buffers.

Single-stage networks make every convolution block-sparse (Section 4); all layers of
a frame use the frame's one execution grid (Section 3.5); each layer's output is a
persistent buffer that keeps transferred blocks from the previous execution
(Section 3.1, Fig. 3); the first frame of a clip runs on every block (Section 4,
BlockCopy configuration). Layers run in network order on one HIP stream.

Backbones: ResNet-18 (basic blocks [2, 2, 2, 2]) and ResNet-50 (bottlenecks
[3, 4, 6, 3], stride on the 3x3 convolution), 7x7/2 stem and 3x3/2 max pooling,
batch norm folded into the convolutions (bc_fold_bn), no classifier. All feature
maps are channels-last bf16 (or fp16). Work per frame: one bc_build_block_index (or an
index handed in, e.g. from bc_sample_execution_grid) and one library call per layer;
nothing runs on the host in between.

Segmentation network (Section 4: a SwiftNet-style single-scale model): the backbone as
encoder, a spatial pyramid pooling module on its stride-32 output (a 1x1 bottleneck;
levels with 8, 4, 2 and 1 rows of bins, each pooled densely from the whole current
bottleneck buffer and projected by a 1x1 convolution, upsampled and concatenated at the
executed blocks, bc_sparse_spp; a 1x1 fuse), then a decoder from stride 32 up to stride
4 in which every level upsamples the coarser decoder feature by two
(bc_sparse_upsample_add), adds a 1x1 projection of the encoder feature at that stride
and blends with a 3x3 convolution; a 1x1 head gives the class scores at stride 4. The
head computes 64 channels per started 64 classes, the first `classes` being the scores.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

from . import bc


@dataclass
class Layer:
    kind: str                  # "conv", "pool", "up" (upsample src by 2, add res) or
                               # "spp" (pyramid pooling; params: grid rows, cl)
    name: str
    src: int                   # producing layer, -1 = the frame
    cin: int
    cout: int
    k: int
    stride: int
    relu: bool = True
    res: int | None = None     # layer whose buffer is added before the ReLU
    params: dict = field(default_factory=dict)

    @property
    def pad(self) -> int:
        return self.k // 2


def build_layers(depth: int) -> list[Layer]:
    """The backbone as a flat list in execution order."""
    if depth == 18:
        blocks, bottleneck = (2, 2, 2, 2), False
    elif depth == 50:
        blocks, bottleneck = (3, 4, 6, 3), True
    else:
        raise ValueError(f"ResNet-{depth} is not provided")
    L = [Layer("conv", "stem", -1, 3, 64, 7, 2),
         Layer("pool", "maxpool", 0, 64, 64, 3, 2, relu=False)]
    cur, ch = 1, 64
    for stage, nblk in enumerate(blocks):
        width = 64 << stage
        out_ch = width * (4 if bottleneck else 1)
        for b in range(nblk):
            stride = 2 if (stage and b == 0) else 1
            tag = f"layer{stage + 1}.{b}"
            shortcut = cur
            if b == 0 and (stride != 1 or ch != out_ch):
                L.append(Layer("conv", tag + ".downsample", cur, ch, out_ch, 1, stride, relu=False))
                shortcut = len(L) - 1
            if bottleneck:
                L.append(Layer("conv", tag + ".conv1", cur, ch, width, 1, 1))
                L.append(Layer("conv", tag + ".conv2", len(L) - 1, width, width, 3, stride))
                L.append(Layer("conv", tag + ".conv3", len(L) - 1, width, out_ch, 1, 1, res=shortcut))
            else:
                L.append(Layer("conv", tag + ".conv1", cur, ch, width, 3, stride))
                L.append(Layer("conv", tag + ".conv2", len(L) - 1, width, out_ch, 3, 1, res=shortcut))
            cur, ch = len(L) - 1, out_ch
    return L


SPP_ROWS = (8, 4, 2, 1)      # rows of the pyramid levels' bin grids


def spp_grid(h: int, w: int, rows: int) -> tuple[int, int]:
    """Bins of a pyramid level with `rows` rows on an h x w map: rows (at most h) by
    rows * w / h rounded half up (1..w), about square bins on wide maps."""
    r = min(rows, h)
    return r, min(w, max(1, (2 * rows * w + h) // (2 * h)))


def build_swiftnet_layers(depth: int = 18, classes: int = 19, width: int = 128) -> list[Layer]:
    """Encoder (the backbone of build_layers) followed by the decoder, in execution
    order: dec.spp.bottleneck (1x1 on the stride-32 output), dec.spp (pyramid pooling,
    concatenating width/4 channels per level after the bottleneck), dec.spp.fuse (1x1
    back to `width`), then per level s = 3, 2, 1 the lateral dec.lat{s} (1x1 on the last
    output of encoder stage s), dec.up{s} (coarser decoder feature upsampled by two plus
    the lateral) and dec.blend{s} (3x3); then dec.logits (1x1, no ReLU)."""
    L = build_layers(depth)
    grow = 4 if depth == 50 else 1
    last = {}
    for i, l in enumerate(L):
        if l.name.startswith("layer"):
            last[int(l.name[len("layer")])] = i          # ends on the stage's last layer

    def add(layer: Layer) -> int:
        L.append(layer)
        return len(L) - 1

    b = add(Layer("conv", "dec.spp.bottleneck", last[4], 512 * grow, width, 1, 1))
    cl = width // 4
    cat = width + len(SPP_ROWS) * cl
    spp = add(Layer("spp", "dec.spp", b, width, cat, 1, 1, params=dict(rows=SPP_ROWS, cl=cl)))
    x = add(Layer("conv", "dec.spp.fuse", spp, cat, width, 1, 1))
    for s in (3, 2, 1):
        lat = add(Layer("conv", f"dec.lat{s}", last[s], (32 << s) * grow, width, 1, 1))
        up = add(Layer("up", f"dec.up{s}", x, width, width, 1, 1, relu=False, res=lat))
        x = add(Layer("conv", f"dec.blend{s}", up, width, width, 3, 1))
    add(Layer("conv", "dec.logits", x, width, 64 * -(-classes // 64), 1, 1, relu=False))
    return L


def default_params(layers: list[Layer], seed0: int = 1000, bn_random: bool = False):
    """He-normal fp32 OIHW weights (seed seed0 + layer position) and batch-norm
    statistics (identity unless bn_random), drawn by the shared input generators; a
    pyramid pooling layer gets one set per level (1x1, cl x cin), in level order."""
    import synth
    out = []

    def one(r, cout, cin, k):
        w = synth.he_normal(r, cout, cin, k, k)
        if bn_random:
            bn = dict(gamma=r.uniform(0.5, 1.5, cout), beta=r.normal(0, 0.1, cout),
                      mean=r.normal(0, 0.1, cout), var=r.uniform(0.5, 1.5, cout))
        else:
            bn = dict(gamma=np.ones(cout), beta=np.zeros(cout), mean=np.zeros(cout), var=np.ones(cout))
        return dict(w=w, **bn)

    for i, l in enumerate(layers):
        r = synth.rng(seed0 + i)
        if l.kind == "conv":
            out.append(one(r, l.cout, l.cin, l.k))
        elif l.kind == "spp":
            out.append(dict(levels=[one(r, l.params["cl"], l.cin, 1) for _ in l.params["rows"]]))
        else:
            out.append(None)
    return out


def device_weights(layers: list[Layer], params, dtype, device):
    """Batch norm folded into each conv (bc_fold_bn) and the weights repacked to the
    channels-last layout in `dtype` (bc_repack_weights), on the device; None for layers
    without weights. A pyramid pooling layer's levels are stacked: weights
    [levels][cl][cin], biases [levels][cl]."""
    dcode = bc.BC_BF16 if dtype == torch.bfloat16 else bc.BC_F16

    def fold(p):
        wf, bf = bc.bc_fold_bn(p["w"], None, p["gamma"], p["beta"], p["mean"], p["var"], 1e-5)
        wr = bc.bc_repack_weights(wf.reshape(p["w"].shape), dcode)
        return torch.from_numpy(wr.view(np.int16)).view(dtype), torch.from_numpy(bf)

    weights, biases = [], []
    for l, p in zip(layers, params):
        if l.kind == "conv":
            w, b = fold(p)
        elif l.kind == "spp":
            parts = [fold(q) for q in p["levels"]]
            w = torch.stack([q[0].reshape(l.params["cl"], l.cin) for q in parts])
            b = torch.stack([q[1] for q in parts])
        else:
            weights.append(None)
            biases.append(None)
            continue
        weights.append(w.to(device).contiguous())
        biases.append(b.to(device).contiguous())
    return weights, biases


def build_policy_layers() -> list[Layer]:
    """The policy network on S_t (32 channels at a quarter of the frame resolution):
    3x3/2 stem to 64 channels, basic blocks of 64, 128 (stride 2) and 256 (stride 2)
    channels with 1x1/2 projections on the strided shortcuts, and a fully convolutional
    head of two 3x3/2 convolutions to one pixel per 128-pixel block (64 channels,
    channel 0 the block's logit)."""
    L = [Layer("conv", "pn.stem", -1, 32, 64, 3, 2)]
    L.append(Layer("conv", "pn.block1.conv1", 0, 64, 64, 3, 1))
    L.append(Layer("conv", "pn.block1.conv2", 1, 64, 64, 3, 1, res=0))
    cur, ch = 2, 64
    for i, width in ((2, 128), (3, 256)):
        L.append(Layer("conv", f"pn.block{i}.downsample", cur, ch, width, 1, 2, relu=False))
        ds = len(L) - 1
        L.append(Layer("conv", f"pn.block{i}.conv1", cur, ch, width, 3, 2))
        L.append(Layer("conv", f"pn.block{i}.conv2", len(L) - 1, width, width, 3, 1, res=ds))
        cur, ch = len(L) - 1, width
    L.append(Layer("conv", "pn.head1", cur, 256, 64, 3, 2))
    L.append(Layer("conv", "pn.head2", len(L) - 1, 64, 64, 3, 2, relu=False))
    return L


class PolicyNet:
    """The policy network's forward pass on the device (Section 3.3, Eq. 2): S_t
    assembled by bc_policy_input, the convolutions on the dense path (every block; each
    layer on a grid of at most 8x8-pixel blocks), P_t by bc_policy_probabilities.
    h, w: frame size; block: block edge in frame pixels (the head ends on that grid)."""

    def __init__(self, h: int, w: int, block: int = 128, classes: int = 19, params=None,
                 dtype=torch.bfloat16, device="cuda", seed0: int = 3000):
        if h % block or w % block or block != 128:
            raise ValueError("the head reduces the frame by 128: blocks of 128 pixels")
        self.layers = build_policy_layers()
        self.classes, self.dtype, self.device = classes, dtype, torch.device(device)
        self.grid = (h // block, w // block)
        params = params if params is not None else default_params(self.layers, seed0)
        self.shapes = layer_shapes(self.layers, h // 4, w // 4)
        self.weights, self.biases = device_weights(self.layers, params, dtype, self.device)
        self.input = torch.empty((1, h // 4, w // 4, 32), dtype=dtype, device=self.device)
        self.buffers = [torch.empty((1, oh, ow, c), dtype=dtype, device=self.device)
                        for (oh, ow, c) in self.shapes]
        self.grids = [(oh // min(8, oh), ow // min(8, ow)) for (oh, ow, _) in self.shapes]
        self.prob = torch.empty((1,) + self.grid, dtype=torch.float32, device=self.device)

    def macs(self) -> float:
        return float(sum(l.cin * l.cout * l.k * l.k * oh * ow
                         for l, (oh, ow, _) in zip(self.layers, self.shapes)))

    def forward(self, frame, state, scores, prev_mask, stream=None):
        """frame, state [1, h, w, 3]; scores [1, h/4, w/4, c] (O_{t-1}); prev_mask uint8
        [1, gh, gw] (A_{t-1}) or None. Returns P_t (self.prob, float32 [1, gh, gw])."""
        bc.bc_policy_input(frame, state, scores, self.classes, prev_mask, self.grid, self.input,
                           stream)
        for i, l in enumerate(self.layers):
            src = self.input if l.src < 0 else self.buffers[l.src]
            res = None if l.res is None else self.buffers[l.res]
            bc.bc_sparse_conv2d((l.k, l.k, l.stride, l.pad, int(l.relu)), src, bc.BC_NHWC,
                                self.weights[i], self.biases[i], res, self.buffers[i],
                                self.grids[i], None, None, stream)
        bc.bc_policy_probabilities(self.buffers[-1], self.prob, stream)
        return self.prob

    # ------------------------------------------------------------------ online update
    def _init_training(self):
        """fp32 master weights ([cout][k][k][cin], the layout the convolutions read),
        RMSprop state and gradient accumulators, and two gradient maps per layer."""
        dev, dt = self.device, self.dtype
        self.master, self.v_w, self.dw, self.v_b, self.db = [], [], [], [], []
        for wt in self.weights:
            m = wt.float().contiguous()
            self.master.append(m)
            self.v_w.append(torch.zeros_like(m))
            self.dw.append(torch.zeros_like(m))
        for b in self.biases:
            self.v_b.append(torch.zeros_like(b))
            self.db.append(torch.zeros_like(b))
        self.gbufs = [[torch.empty((1, oh, ow, c), dtype=dt, device=dev) for _ in range(2)]
                      for (oh, ow, c) in self.shapes]

    def backward(self, reward, mask, prob, stream=None):
        """Adds the gradients of L = -sum_b R_b log pi(a_b) at the last forward pass to
        self.dw / self.db. reward, prob float32 [1, gh, gw]; mask uint8 (the executed
        grid a_b)."""
        if not hasattr(self, "master"):
            self._init_training()
        last = len(self.layers) - 1
        cur = {last: self.gbufs[last][0]}
        bc.bc_policy_logit_grad(reward, mask, prob, cur[last], stream)
        for li in range(last, -1, -1):
            l = self.layers[li]
            gp = cur.pop(li)                          # complete: every consumer came later
            if l.relu:
                bc.bc_grad_combine(gp, None, self.buffers[li], gp, stream)
            geom = (l.k, l.k, l.stride, l.pad, 0)
            src = self.input if l.src < 0 else self.buffers[l.src]
            bc.bc_conv2d_weight_grad(geom, src, gp, self.dw[li], self.db[li], stream)
            if l.src >= 0:
                acc = cur.get(l.src)
                out = self.gbufs[l.src][1] if acc is self.gbufs[l.src][0] else self.gbufs[l.src][0]
                bc.bc_conv2d_input_grad(geom, gp, self.weights[li], acc, out, stream)
                cur[l.src] = out
            if l.res is not None:
                acc = cur.get(l.res)
                if acc is None:
                    # the shortcut passes gp on unchanged; layer li's buffer is free from
                    # here on and has l.res's shape, so it takes the sum in place
                    cur[l.res] = gp
                else:
                    bc.bc_grad_combine(acc, gp, None, acc, stream)

    def update(self, lr=1e-4, alpha=0.99, eps=1e-8, weight_decay=1e-3, stream=None):
        """One RMSprop step on every weight and bias with the accumulated gradients (which
        it resets); the 16-bit weights the convolutions read are rewritten."""
        params = []
        for i in range(len(self.layers)):
            params.append((self.master[i], self.v_w[i], self.dw[i], self.weights[i]))
            params.append((self.biases[i], self.v_b[i], self.db[i], None))
        bc.bc_rmsprop_step_many(params, lr, alpha, eps, weight_decay, stream)

    def train_step(self, reward, mask, prob, stream=None, **rmsprop):
        """The online update of Section 4: backward pass at the last forward pass, then one
        RMSprop step."""
        self.backward(reward, mask, prob, stream)
        self.update(stream=stream, **rmsprop)


def layer_shapes(layers: list[Layer], h: int, w: int) -> list[tuple[int, int, int]]:
    """(out_h, out_w, out_c) of every layer for an h x w frame (the dense conv formula)."""
    shapes = []
    for l in layers:
        ih, iw = (h, w) if l.src < 0 else shapes[l.src][:2]
        if l.kind == "up":
            shapes.append((2 * ih, 2 * iw, l.cout))
            continue
        shapes.append(((ih + 2 * l.pad - l.k) // l.stride + 1,
                       (iw + 2 * l.pad - l.k) // l.stride + 1, l.cout))
    return shapes


def conv_algo_bytes(layers: list[Layer], shapes, grid, active: int, esize: int = 2):
    """Algorithmic HBM bytes of each convolution with `active` of the grid's blocks
    executed: every element of the active blocks' input halo tiles read once, the
    weights read once, the active output blocks (and residual blocks) read/written
    once. Returns a list aligned with `layers` (None for non-conv layers)."""
    gh, gw = grid
    out = []
    for l, (oh, ow, co) in zip(layers, shapes):
        if l.kind != "conv":
            out.append(None)
            continue
        bh, bw = oh // gh, ow // gw
        th, tw = (bh - 1) * l.stride + l.k, (bw - 1) * l.stride + l.k
        halo = active * th * tw * l.cin * esize
        wts = l.cout * l.k * l.k * l.cin * esize + l.cout * 4
        outb = active * bh * bw * co * esize
        out.append(halo + wts + outb * (2 if l.res is not None else 1))
    return out


class SparseResNet:
    """ResNet backbone executed block-sparsely frame by frame.

    h, w: frame size; block: block edge in image pixels (the grid is h/block x
    w/block for every layer, each layer's block edge is block / its stride).
    """

    def __init__(self, depth: int, h: int, w: int, block: int = 128, params=None,
                 dtype=torch.bfloat16, device="cuda", seed0: int = 1000, bn_random: bool = False,
                 layers: list[Layer] | None = None):
        if h % block or w % block or block % 32:
            raise ValueError("frame size must be a multiple of the block size, and the block "
                             "size a multiple of 32 (the backbone's total stride)")
        self.layers = layers if layers is not None else build_layers(depth)
        self.h, self.w, self.block = h, w, block
        self.grid = (h // block, w // block)
        self.dtype, self.device = dtype, torch.device(device)
        params = params if params is not None else default_params(self.layers, seed0, bn_random)
        self.shapes = layer_shapes(self.layers, h, w)
        self.weights, self.biases = device_weights(self.layers, params, dtype, self.device)
        self.buffers = [torch.empty((1, oh, ow, c), dtype=dtype, device=self.device)
                        for (oh, ow, c) in self.shapes]
        self.handles = [bc.Buffer(t, bc.BC_NHWC) for t in self.buffers]
        # pyramid pooling: each level's bin grid on its map, and the level buffer the
        # library rewrites every frame
        self.spp = {}
        for i, l in enumerate(self.layers):
            if l.kind == "spp":
                ih, iw, _ = self.shapes[l.src]
                bins = [spp_grid(ih, iw, r) for r in l.params["rows"]]
                lv = torch.empty((1, sum(a * b for a, b in bins), l.params["cl"]), dtype=dtype,
                                 device=self.device)
                self.spp[i] = (bins, lv)
        nblk = self.grid[0] * self.grid[1]
        self.idx = torch.zeros(nblk, dtype=torch.int32, device=self.device)
        self.count = torch.zeros(1, dtype=torch.int32, device=self.device)
        self.mask = torch.zeros((1,) + self.grid, dtype=torch.uint8, device=self.device)
        self.pairs = self._find_pairs()
        self.pair_launches = True

    # ------------------------------------------------------------------
    def conv_flops(self, active_blocks: int) -> float:
        """Algorithmic FLOPs of the convolutions for one frame with that many active blocks."""
        nblk = self.grid[0] * self.grid[1]
        tot = 0.0
        for l, (oh, ow, c) in zip(self.layers, self.shapes):
            if l.kind == "conv":
                tot += 2.0 * l.cin * l.cout * l.k * l.k * oh * ow * active_blocks / nblk
        return tot

    def invalidate(self):
        """Start of a new clip: the next frame must be a full one."""
        for hd in self.handles:
            hd.invalidate()

    def set_mask(self, mask):
        """Copy an execution grid ([1, gh, gw] uint8, host or device) into the frame's mask."""
        m = torch.as_tensor(np.asarray(mask, np.uint8) if not torch.is_tensor(mask) else mask)
        self.mask.copy_(m.reshape(self.mask.shape), non_blocking=False)

    def frame(self, x, sparse: bool = True, stream=None, index=None):
        """Run one frame. x: [1, h, w, 3] channels-last on the device. sparse=False runs
        every block (first frame of a clip); sparse=True uses the grid in self.mask, or
        the device (idx, count) pair `index` if given (then self.mask is not read)."""
        if sparse and index is not None:
            idx, cnt = index
        elif sparse:
            bc.bc_build_block_index(self.mask, 1, self.grid, self.idx, self.count, stream=stream)
            idx, cnt = self.idx, self.count
        else:
            idx = cnt = None
        done = set()
        for i in range(len(self.layers)):
            if i in done:
                continue
            j = self.pairs.get(i) if self.pair_launches else None
            if j is None:
                self.run_layer(i, x, idx, cnt, stream)
            else:
                self.run_pair(i, j, x, idx, cnt, stream)
                done.add(j)
        return self.buffers[-1]

    def _find_pairs(self) -> dict[int, int]:
        """{i: j}: layer j > i runs in one launch with layer i, at i's turn. Both are 1x1
        convolutions (j at stride 1) and independent: j reads only layers before i (so
        moving it forward changes nothing it reads) and nothing between them reads j,
        which only later layers can. Found greedily: a block's shortcut projection with
        its branch's first convolution; a decoder's lateral projections with each other."""
        L, out, taken = self.layers, {}, set()

        def one_by_one(l):
            return l.kind == "conv" and l.k == 1

        for i, a in enumerate(L):
            if i in taken or not one_by_one(a):
                continue
            for j in range(i + 1, len(L)):
                b = L[j]
                if (j not in taken and one_by_one(b) and b.stride == 1 and b.src < i
                        and (b.res is None or b.res < i)):
                    out[i] = j
                    taken.update((i, j))
                    break
        return out

    def _call(self, i, x):
        l = self.layers[i]
        src = x if l.src < 0 else self.buffers[l.src]
        res = None if l.res is None else self.buffers[l.res]
        return ((l.k, l.k, l.stride, l.pad, int(l.relu)), src, bc.BC_NHWC, self.weights[i],
                self.biases[i], res, self.buffers[i])

    def run_pair(self, i, j, x, idx, cnt, stream=None):
        """Layers i and j (see _find_pairs) through one library call."""
        bc.bc_sparse_conv2d_pair(self._call(i, x), self._call(j, x), self.grid, idx, cnt, stream)

    def run_layer(self, i, x, idx, cnt, stream=None):
        l = self.layers[i]
        src = x if l.src < 0 else self.buffers[l.src]
        out = self.buffers[i]
        if l.kind == "pool":
            bc.bc_sparse_maxpool2d((l.k, l.k, l.stride, l.pad, 0), src, bc.BC_NHWC, out, self.grid,
                                   idx, cnt, stream)
        elif l.kind == "up":
            bc.bc_sparse_upsample_add(src, bc.BC_NHWC, self.buffers[l.res], out, self.grid,
                                      int(l.relu), idx, cnt, stream)
        elif l.kind == "spp":
            bins, lv = self.spp[i]
            bc.bc_sparse_spp(src, bc.BC_NHWC, [a for a, _ in bins], [b for _, b in bins],
                             l.params["cl"], self.weights[i], self.biases[i], lv, out, self.grid,
                             idx, cnt, stream)
        else:
            res = None if l.res is None else self.buffers[l.res]
            bc.bc_sparse_conv2d((l.k, l.k, l.stride, l.pad, int(l.relu)), src, bc.BC_NHWC,
                                self.weights[i], self.biases[i], res, out, self.grid, idx, cnt,
                                stream)


class SparseSwiftNet(SparseResNet):
    """SwiftNet-style segmentation network (encoder = ResNet backbone, decoder of
    build_swiftnet_layers) executed block-sparsely frame by frame. `logits` is the
    persistent stride-4 score buffer [1, h/4, w/4, 64*ceil(classes/64)] whose first
    `classes` channels are the class scores."""

    def __init__(self, depth: int, h: int, w: int, block: int = 128, classes: int = 19,
                 width: int = 128, **kw):
        self.classes = classes
        super().__init__(depth, h, w, block, layers=build_swiftnet_layers(depth, classes, width), **kw)

    @property
    def logits(self):
        return self.buffers[-1]
