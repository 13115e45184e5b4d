"""Seeded synthetic workloads for the recomputation DP (inputs only).

This module is shared by the GPU path and the oracle, so it holds no part
of the method's arithmetic: it builds a DAG (successor CSR over node ids
0..n-1) and the per-node integer costs T_v (forward time) and M_v (memory
size) that Section 2 of the paper attaches to every intermediate node,
plus the budget B, family mode and objective of each benchmark case.

Graph model (Section 2): a node is an intermediate variable of the
network; an edge (v, w) means v is directly needed to compute w; input
nodes and parameters are not nodes.  The paper's own experiments run on
real ResNet, DenseNet and U-Net graphs (Section 5); the CNN-shaped
generators below stand in for them.  Costs of CNN-shaped graphs: M_v is
the fp32 activation size of the op's output in MiB (rounded up) at the
stated batch, T_v the op's forward cost in MFLOPs (rounded up, at least
1, because Section 2 requires T_v > 0 and M_v > 0).

FLOP conventions: conv 2*N*Cin*Cout*k*k*Hout*Wout; transposed conv 2x2
stride 2: 2*N*Cin*Cout*4*Hin*Win; batch norm 4 per output element; ReLU
and add 1 per output element; max/avg pool k*k per output element;
global pool 1 per input element; concat and crop 0 (clamped to 1); fully
connected 2*N*in*out.

Random draws use Python's ``random.Random(seed)`` (Mersenne Twister).
"""

from __future__ import annotations

import random
from dataclasses import dataclass, field

MIB = 1 << 20

__all__ = [
    "Graph", "Case", "chain", "layered", "ladder", "resnet50", "densenet121",
    "unet", "random_dag", "antichain", "CASES", "case", "PAPER_COST_CONVENTION", "paper_costs",
]


@dataclass
class Graph:
    """A DAG as successor lists plus integer costs.

    ``succ[v]`` lists the nodes w with an edge v -> w.  ``T`` and ``M`` are
    the per-node forward time and memory size (both >= 1).  ``names`` and
    ``ops`` are labels only.
    """

    n: int
    succ: list
    T: list
    M: list
    names: list = field(default_factory=list)
    ops: list = field(default_factory=list)

    def csr(self):
        """Successor CSR ``(row_ptr, col_idx)`` as plain int lists."""
        row_ptr = [0]
        col_idx = []
        for v in range(self.n):
            col_idx.extend(self.succ[v])
            row_ptr.append(len(col_idx))
        return row_ptr, col_idx

    @property
    def num_edges(self):
        return sum(len(s) for s in self.succ)

    def relabel(self, perm):
        """Return the same graph with node v renamed perm[v]."""
        n = self.n
        succ = [None] * n
        T = [0] * n
        M = [0] * n
        names = [""] * n
        ops = [""] * n
        for v in range(n):
            pv = perm[v]
            succ[pv] = sorted(perm[w] for w in self.succ[v])
            T[pv] = self.T[v]
            M[pv] = self.M[v]
            if self.names:
                names[pv] = self.names[v]
            if self.ops:
                ops[pv] = self.ops[v]
        return Graph(n, succ, T, M, names if self.names else [], ops if self.ops else [])


@dataclass
class Case:
    """One benchmark case: a graph plus family mode, budget and objective."""

    name: str
    graph: Graph
    mode: str          # "exact" or "pruned"
    B: int
    objective: str     # "tc" or "mc"
    note: str = ""


# ----------------------------------------------------------------------------
# Small random graphs


def chain(n=16, seed=0, tmax=10, mmax=8):
    """Linear chain v0 -> v1 -> ... -> v(n-1); per node T ~ U{1..tmax}
    then M ~ U{1..mmax} from ``random.Random(seed)``."""
    rng = random.Random(seed)
    T, M = [], []
    for _ in range(n):
        T.append(rng.randint(1, tmax))
        M.append(rng.randint(1, mmax))
    succ = [[v + 1] if v + 1 < n else [] for v in range(n)]
    return Graph(n, succ, T, M, [f"v{v}" for v in range(n)], ["op"] * n)


def layered(layers=8, width=3, seed=0, tmax=100, mmax=64):
    """Random layered DAG.  Node ids run layer by layer.  For every node of
    layer l >= 1 (in id order): draw k ~ U{1..3} and k distinct predecessors
    from layer l-1; for l >= 2 also one skip predecessor drawn uniformly from
    all nodes of layers < l-1.  Then, per node in id order, T ~ U{1..tmax}
    and M ~ U{1..mmax}."""
    rng = random.Random(seed)
    n = layers * width
    preds = [[] for _ in range(n)]
    for l in range(1, layers):
        prev = list(range((l - 1) * width, l * width))
        for v in range(l * width, (l + 1) * width):
            k = rng.randint(1, min(3, width))
            ps = rng.sample(prev, k)
            if l >= 2:
                ps.append(rng.randrange(0, (l - 1) * width))
            preds[v] = sorted(set(ps))
    T, M = [], []
    for _ in range(n):
        T.append(rng.randint(1, tmax))
        M.append(rng.randint(1, mmax))
    succ = [[] for _ in range(n)]
    for v in range(n):
        for p in preds[v]:
            succ[p].append(v)
    succ = [sorted(s) for s in succ]
    return Graph(n, succ, T, M, [f"l{v // width}_{v % width}" for v in range(n)], ["op"] * n)


def ladder(length=20, seed=0, tmax=100, mmax=64, cross_every=2):
    """Two chains a_0..a_{L-1}, b_0..b_{L-1} with a cross edge a_i -> b_i for
    every i with i % cross_every == cross_every - 1 (odd i for the default).
    Node ids: a_i = 2i, b_i = 2i + 1.  Per node in id order T ~ U{1..tmax}
    then M ~ U{1..mmax}."""
    rng = random.Random(seed)
    n = 2 * length
    succ = [[] for _ in range(n)]
    for i in range(length):
        a, b = 2 * i, 2 * i + 1
        if i + 1 < length:
            succ[a].append(2 * (i + 1))
            succ[b].append(2 * (i + 1) + 1)
        if i % cross_every == cross_every - 1:
            succ[a].append(b)
    T, M = [], []
    for _ in range(n):
        T.append(rng.randint(1, tmax))
        M.append(rng.randint(1, mmax))
    names = []
    for i in range(length):
        names += [f"a{i}", f"b{i}"]
    return Graph(n, [sorted(s) for s in succ], T, M, names, ["op"] * n)


def random_dag(n, p, seed, tmax=10, mmax=8, shuffle_ids=True):
    """Random DAG: for a hidden order u0 < u1 < ..., edge u_i -> u_j (i < j)
    with probability p.  With ``shuffle_ids`` the node ids are a random
    permutation of that order, so ids need not be topological."""
    rng = random.Random(seed)
    succ = [[] for _ in range(n)]
    for i in range(n):
        for j in range(i + 1, n):
            if rng.random() < p:
                succ[i].append(j)
    T = [rng.randint(1, tmax) for _ in range(n)]
    M = [rng.randint(1, mmax) for _ in range(n)]
    g = Graph(n, succ, T, M)
    if shuffle_ids:
        perm = list(range(n))
        rng.shuffle(perm)
        g = g.relabel(perm)
    return g


def antichain(n, seed=0, tmax=10, mmax=8):
    """n isolated nodes (no edges): every subset is a lower set."""
    rng = random.Random(seed)
    T = [rng.randint(1, tmax) for _ in range(n)]
    M = [rng.randint(1, mmax) for _ in range(n)]
    return Graph(n, [[] for _ in range(n)], T, M)


# ----------------------------------------------------------------------------
# CNN-shaped graphs


def _ceil_div(a, b):
    return -(-a // b)


class _Net:
    """Builder of a CNN-shaped op graph; nodes get ids in creation order."""

    def __init__(self, batch, bytes_per_elem=4):
        self.N = batch
        self.bpe = bytes_per_elem
        self.preds = []
        self.shape = []     # (C, H, W) of each node's output
        self.T = []
        self.M = []
        self.names = []
        self.ops = []

    def _add(self, name, op, preds, shape, flops):
        c, h, w = shape
        self.preds.append(list(preds))
        self.shape.append(shape)
        self.M.append(max(1, _ceil_div(self.bpe * self.N * c * h * w, MIB)))
        self.T.append(max(1, _ceil_div(flops, 10 ** 6)))
        self.names.append(name)
        self.ops.append(op)
        return len(self.preds) - 1

    def conv(self, name, x, cin_shape, cout, k, stride=1, pad=0):
        cin, h, w = cin_shape
        ho = (h + 2 * pad - k) // stride + 1
        wo = (w + 2 * pad - k) // stride + 1
        flops = 2 * self.N * cin * cout * k * k * ho * wo
        preds = [] if x is None else [x]
        return self._add(name, "conv", preds, (cout, ho, wo), flops)

    def upconv(self, name, x, cout):
        cin, h, w = self.shape[x]
        flops = 2 * self.N * cin * cout * 4 * h * w
        return self._add(name, "upconv", [x], (cout, 2 * h, 2 * w), flops)

    def _elementwise(self, name, op, preds, per_elem):
        c, h, w = self.shape[preds[0]]
        return self._add(name, op, preds, (c, h, w), per_elem * self.N * c * h * w)

    def bn(self, name, x):
        return self._elementwise(name, "bn", [x], 4)

    def relu(self, name, x):
        return self._elementwise(name, "relu", [x], 1)

    def add(self, name, xs):
        return self._elementwise(name, "add", xs, 1)

    def pool(self, name, x, k, stride, pad=0, kind="maxpool"):
        c, h, w = self.shape[x]
        ho = (h + 2 * pad - k) // stride + 1
        wo = (w + 2 * pad - k) // stride + 1
        return self._add(name, kind, [x], (c, ho, wo), k * k * self.N * c * ho * wo)

    def gap(self, name, x):
        c, h, w = self.shape[x]
        return self._add(name, "gap", [x], (c, 1, 1), self.N * c * h * w)

    def fc(self, name, x, out):
        c, h, w = self.shape[x]
        fin = c * h * w
        return self._add(name, "fc", [x], (out, 1, 1), 2 * self.N * fin * out)

    def concat(self, name, xs):
        c = sum(self.shape[x][0] for x in xs)
        _, h, w = self.shape[xs[0]]
        return self._add(name, "concat", xs, (c, h, w), 0)

    def crop(self, name, x, h, w):
        c = self.shape[x][0]
        return self._add(name, "crop", [x], (c, h, w), 0)

    def graph(self):
        n = len(self.preds)
        succ = [[] for _ in range(n)]
        for v in range(n):
            for p in self.preds[v]:
                succ[p].append(v)
        return Graph(n, [sorted(set(s)) for s in succ], list(self.T), list(self.M),
                     list(self.names), list(self.ops))


def resnet50(batch=32, image=224):
    """ResNet-50-shaped DAG: stem conv7x7/2-BN-ReLU-maxpool3x3/2, then 16
    bottleneck blocks in stages [3, 4, 6, 3] (widths 64..512, expansion 4;
    stride 2 in the 3x3 conv of the first block of stages 2-4).  Block:
    conv1x1-BN-ReLU, conv3x3-BN-ReLU, conv1x1-BN; the first block of each
    stage adds a projection conv1x1-BN on the block input; then add and
    ReLU.  Head: global average pool and FC 2048 -> 1000.  174 nodes."""
    net = _Net(batch)
    x = net.conv("conv1", None, (3, image, image), 64, 7, 2, 3)
    x = net.bn("bn1", x)
    x = net.relu("relu1", x)
    x = net.pool("maxpool", x, 3, 2, 1)
    cin = 64
    for s, (nblocks, width) in enumerate(zip([3, 4, 6, 3], [64, 128, 256, 512])):
        for b in range(nblocks):
            stride = 2 if (b == 0 and s > 0) else 1
            pre = f"s{s + 1}b{b + 1}"
            inp = x
            ishape = net.shape[inp]
            y = net.conv(pre + ".conv1", inp, ishape, width, 1)
            y = net.bn(pre + ".bn1", y)
            y = net.relu(pre + ".relu1", y)
            y = net.conv(pre + ".conv2", y, net.shape[y], width, 3, stride, 1)
            y = net.bn(pre + ".bn2", y)
            y = net.relu(pre + ".relu2", y)
            y = net.conv(pre + ".conv3", y, net.shape[y], 4 * width, 1)
            y = net.bn(pre + ".bn3", y)
            if b == 0:
                sc = net.conv(pre + ".proj", inp, ishape, 4 * width, 1, stride)
                sc = net.bn(pre + ".projbn", sc)
            else:
                sc = inp
            x = net.add(pre + ".add", [y, sc])
            x = net.relu(pre + ".relu", x)
            cin = 4 * width
    x = net.gap("gap", x)
    net.fc("fc", x, 1000)
    return net.graph()


def densenet121(batch=32, image=224, growth=32, blocks=(6, 12, 24, 16), bn_size=4):
    """DenseNet-121-shaped DAG (growth rate 32): stem conv7x7/2-BN-ReLU-
    maxpool3x3/2; four dense blocks of 6/12/24/16 layers.  Layer l of a
    block reads the concat of the block input and the outputs of layers
    1..l-1 (layer 1 reads the block input directly), then BN-ReLU-
    conv1x1(4k)-BN-ReLU-conv3x3(k).  Transitions: concat of the block,
    BN-ReLU-conv1x1(C/2)-avgpool2x2.  Head: concat, BN, ReLU, global
    average pool, FC -> 1000.  426 nodes."""
    net = _Net(batch)
    x = net.conv("conv0", None, (3, image, image), 64, 7, 2, 3)
    x = net.bn("bn0", x)
    x = net.relu("relu0", x)
    x = net.pool("pool0", x, 3, 2, 1)
    for bi, nl in enumerate(blocks):
        block_in = x
        outs = []
        for l in range(nl):
            pre = f"b{bi + 1}l{l + 1}"
            if l == 0:
                inp = block_in
            else:
                inp = net.concat(pre + ".cat", [block_in] + outs)
            y = net.bn(pre + ".bn1", inp)
            y = net.relu(pre + ".relu1", y)
            y = net.conv(pre + ".conv1", y, net.shape[y], bn_size * growth, 1)
            y = net.bn(pre + ".bn2", y)
            y = net.relu(pre + ".relu2", y)
            y = net.conv(pre + ".conv2", y, net.shape[y], growth, 3, 1, 1)
            outs.append(y)
        cat = net.concat(f"b{bi + 1}.cat", [block_in] + outs)
        if bi + 1 < len(blocks):
            pre = f"t{bi + 1}"
            y = net.bn(pre + ".bn", cat)
            y = net.relu(pre + ".relu", y)
            y = net.conv(pre + ".conv", y, net.shape[y], net.shape[cat][0] // 2, 1)
            x = net.pool(pre + ".pool", y, 2, 2, kind="avgpool")
        else:
            y = net.bn("norm5", cat)
            y = net.relu("relu5", y)
            y = net.gap("gap", y)
            net.fc("fc", y, 1000)
    return net.graph()


def unet(batch=8, image=572, base=64, depth=4):
    """U-Net-shaped DAG with valid 3x3 convolutions: four encoder levels of
    conv-ReLU-conv-ReLU + maxpool2x2 (channels 64..512), a bottom level of
    conv-ReLU-conv-ReLU at 1024 channels, four decoder levels of
    upconv2x2 -> crop(skip) -> concat -> conv-ReLU-conv-ReLU, and a final
    conv1x1 to 2 classes.  Input 1 x 572 x 572.  53 nodes."""
    net = _Net(batch)
    shape = (1, image, image)
    x = None
    skips = []
    c = base
    for lvl in range(depth):
        pre = f"enc{lvl + 1}"
        x = net.conv(pre + ".conv1", x, shape, c, 3)
        x = net.relu(pre + ".relu1", x)
        x = net.conv(pre + ".conv2", x, net.shape[x], c, 3)
        x = net.relu(pre + ".relu2", x)
        skips.append(x)
        x = net.pool(pre + ".pool", x, 2, 2)
        shape = net.shape[x]
        c *= 2
    x = net.conv("bottom.conv1", x, net.shape[x], c, 3)
    x = net.relu("bottom.relu1", x)
    x = net.conv("bottom.conv2", x, net.shape[x], c, 3)
    x = net.relu("bottom.relu2", x)
    for lvl in reversed(range(depth)):
        pre = f"dec{lvl + 1}"
        c //= 2
        up = net.upconv(pre + ".up", x, c)
        _, h, w = net.shape[up]
        cr = net.crop(pre + ".crop", skips[lvl], h, w)
        cat = net.concat(pre + ".cat", [cr, up])
        x = net.conv(pre + ".conv1", cat, net.shape[cat], c, 3)
        x = net.relu(pre + ".relu1", x)
        x = net.conv(pre + ".conv2", x, net.shape[x], c, 3)
        x = net.relu(pre + ".relu2", x)
    net.conv("final", x, net.shape[x], 2, 1)
    return net.graph()


# ----------------------------------------------------------------------------
# The benchmark cases (six graphs: the fifth workload has two)

PAPER_COST_CONVENTION = "T_v = 10 for conv, 1 otherwise (Section 3)"


def paper_costs(g):
    """The same graph with the forward times of the paper's experiments: T_v
    = 10 for convolution nodes (transposed ones included) and 1 for every
    other node (end of Section 3); memory sizes unchanged."""
    T = [10 if op in ("conv", "upconv") else 1 for op in g.ops]
    return Graph(g.n, [list(x) for x in g.succ], T, list(g.M), list(g.names), list(g.ops))


def _cases():
    return {
        "chain16": lambda: Case("chain16", chain(16, 0), "exact", 64, "tc",
                                "16-node chain, exact family, B=64"),
        "layered24": lambda: Case("layered24", layered(8, 3, 0), "exact", 256, "tc",
                                  "8x3 random layered DAG, exact family, B=256"),
        "resnet50": lambda: Case("resnet50", resnet50(32, 224), "pruned", 4096, "tc",
                                 "ResNet-50 shape, batch 32, 224^2, pruned family, B=4096"),
        "densenet121": lambda: Case("densenet121", densenet121(32, 224), "pruned", 4096, "tc",
                                    "DenseNet-121 shape, batch 32, 224^2, pruned family, B=4096"),
        "unet": lambda: Case("unet", unet(8, 572), "pruned", 16384, "tc",
                             "U-Net shape, batch 8, 572^2, pruned family, B=16384"),
        "ladder40": lambda: Case("ladder40", ladder(20, 0), "exact", 1024, "tc",
                                 "2x20 ladder, cross edge every 2 nodes, exact family, B=1024"),
        "resnet50_t10": lambda: Case("resnet50_t10", paper_costs(resnet50(32, 224)), "pruned",
                                     4096, "tc", "ResNet-50 shape with T_v = 10 (conv) / 1, "
                                     "pruned family, B=4096"),
        "densenet121_t10": lambda: Case("densenet121_t10", paper_costs(densenet121(32, 224)),
                                        "pruned", 4096, "tc", "DenseNet-121 shape with T_v = 10 "
                                        "(conv) / 1, pruned family, B=4096"),
        "unet_t10": lambda: Case("unet_t10", paper_costs(unet(8, 572)), "pruned", 16384, "tc",
                                 "U-Net shape with T_v = 10 (conv) / 1, pruned family, B=16384"),
    }


CASES = list(_cases().keys())


def case(name):
    """Build the named benchmark case."""
    return _cases()[name]()
