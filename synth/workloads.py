"""The five benchmark workloads: sizes, synthetic-gradient recipes and the
per-tensor layouts of the public model shapes they imitate.

Input description only.  Row counts follow the paper's definitions: the
m x n view has m = ceil(d / n) rows (Eq. (3)) and K = ceil(mu * m) rows are
kept (Alg. 1's input line).  The model layouts are public architecture shapes
(parameter tensors in their usual order); no trained weights or datasets are
involved.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace


def resnet18_views() -> list[tuple[int, int]]:
    """torchvision ResNet-18 (ImageNet head) parameters, in order, as 2-D views:
    convolution kernels as out x (in*kh*kw), the fc weight as out x in, and
    1-D tensors (batch-norm weights and biases, fc bias) as one row."""
    views = [(64, 3 * 7 * 7), (1, 64), (1, 64)]  # conv1, bn1 weight, bn1 bias
    cin = 64
    for cout in (64, 128, 256, 512):
        for block in range(2):
            first_in = cin if block == 0 else cout
            views += [(cout, first_in * 9), (1, cout), (1, cout), (cout, cout * 9), (1, cout),
                      (1, cout)]
            if block == 0 and cout != cin:
                views += [(cout, cin), (1, cout), (1, cout)]  # downsample conv 1x1 + bn
        cin = cout
    views += [(1000, 512), (1, 1000)]  # fc weight, fc bias
    return views


def gpt2_small_views() -> list[tuple[int, int]]:
    """GPT-2 small parameters (embeddings, 12 blocks, final LayerNorm) in their
    stored shapes; the block projections are stored in x out; 1-D tensors as
    one row."""
    h = 768
    views = [(50257, h), (1024, h)]
    for _ in range(12):
        views += [(1, h), (1, h), (h, 3 * h), (1, 3 * h), (h, h), (1, h), (1, h), (1, h),
                  (h, 4 * h), (1, 4 * h), (4 * h, h), (1, h)]
    views += [(1, h), (1, h)]
    return views


def tinyllama_views() -> list[tuple[int, int]]:
    """TinyLlama-1.1B: hidden 2048, MLP 5632, 4 KV heads of 64, 22 blocks,
    untied lm_head; weights out x in, RMSNorm weights as one row."""
    h, f, kv = 2048, 5632, 256
    views = [(32000, h)]
    for _ in range(22):
        views += [(h, h), (kv, h), (kv, h), (h, h), (f, h), (f, h), (h, f), (1, h), (1, h)]
    views += [(1, h), (32000, h)]
    return views


def resnet18_tensors() -> list[int]:
    """ResNet-18 parameter sizes, in order."""
    return [r * c for r, c in resnet18_views()]


def gpt2_small_tensors() -> list[int]:
    """GPT-2 small parameter sizes, in order."""
    return [r * c for r, c in gpt2_small_views()]


def tinyllama_tensors() -> list[int]:
    """TinyLlama-1.1B parameter sizes, in order."""
    return [r * c for r, c in tinyllama_views()]


def llama7b_tensors() -> list[int]:
    """Llama-7B parameters in an order that makes each bucket a contiguous
    block of rows at n = 4096: embedding, 32 blocks of matrices, lm_head, then
    the 65 norm vectors."""
    h, f = 4096, 11008
    sizes = [32000 * h]
    for _ in range(32):
        sizes += [h * h] * 4 + [f * h, f * h, h * f]
    sizes += [32000 * h]
    sizes += [h] * 65
    return sizes


@dataclass
class Workload:
    name: str
    d: int
    N: int
    grad_dtype: str          # "f32" or "bf16"
    steps: int
    eta: float
    mu: float
    n: int
    r: int
    data_seed: int
    sketch_seed: int
    family: int              # 0: scale*(m_j + noise*e_ij); 1: Student-t mix
    noise: float = 0.0
    scale_sigma: float = 1.0  # LogNormal(0, scale_sigma) scales
    per_coord_scale: bool = False
    tensors: list = field(default_factory=list)
    boost: float = 1.0
    boost_frac: float = 0.0
    corr: float = 0.0        # family 1: cross-worker correlation
    buckets_from_tensors: bool = False
    views: list = field(default_factory=list)  # per-tensor mode: [(rows, cols)]
    description: str = ""

    @property
    def per_tensor(self) -> bool:
        return bool(self.views)

    @property
    def m(self) -> int:
        if self.per_tensor:
            return sum(r for r, _ in self.views)
        return -(-self.d // self.n)

    def tensor_views(self):
        """Per-tensor mode: [(rows, cols, K)] with K = ceil(mu * rows) for a
        matrix and the whole tensor for a one-row (1-D) tensor, which the
        paper's experiments leave uncompressed."""
        return [(r, c, r if r == 1 else math.ceil(self.mu * r)) for r, c in self.views]

    @property
    def bytes_per_grad(self) -> int:
        return 2 if self.grad_dtype == "bf16" else 4

    def buckets(self):
        """(row_begin[nb+1], K[nb]) or None for one global selection."""
        if not self.buckets_from_tensors:
            return None
        # embedding, one bucket per block, lm_head, and the dense norm bucket
        h = self.n
        begin, ks = [0], []
        rows_embed = 32000
        rows_block = (4 * h * h + 3 * 11008 * h) // h
        spans = [rows_embed] + [rows_block] * 32 + [rows_embed]
        for rows in spans:
            begin.append(begin[-1] + rows)
            ks.append(math.ceil(self.mu * rows))
        norm_rows = self.m - begin[-1]
        begin.append(self.m)
        ks.append(norm_rows)  # 1-D norm vectors are not compressed (kept dense)
        return begin, ks

    def K_rows(self) -> int:
        """Selected rows per step (total over buckets or tensors)."""
        if self.per_tensor:
            return sum(min(k, r) for r, _, k in self.tensor_views())
        b = self.buckets()
        if b is None:
            return min(self.m, math.ceil(self.mu * self.m))
        begin, ks = b
        return sum(min(k, begin[i + 1] - begin[i]) for i, k in enumerate(ks))

    def K_global(self) -> int:
        if self.buckets_from_tensors or self.per_tensor:
            return 0
        return math.ceil(self.mu * self.m)

    def payload_elems(self) -> int:
        """Elements of the aggregated payload per step."""
        if self.per_tensor:
            return sum(min(k, r) * c for r, c, k in self.tensor_views())
        return self.K_rows() * self.n


WORKLOADS = {
    "tiny": Workload(
        "tiny", d=1_048_576, N=4, grad_dtype="f32", steps=10, eta=0.1, mu=0.01, n=256, r=4,
        data_seed=1001, sketch_seed=2001, family=0, noise=0.3, scale_sigma=1.0,
        per_coord_scale=True,
        description="d=1,048,576 fp32, N=4; per-coordinate LogNormal(0,1) scale shared by "
                    "workers; g=s*(m+0.3e), m,e~N(0,1) fresh per step"),
    "resnet18": Workload(
        "resnet18", d=11_689_512, N=8, grad_dtype="f32", steps=50, eta=0.1, mu=0.01, n=512, r=4,
        data_seed=1002, sketch_seed=2002, family=0, noise=0.5, scale_sigma=1.5,
        tensors=resnet18_tensors(), boost=20.0, boost_frac=0.001,
        description="ResNet-18 layout (62 tensors), per-tensor LogNormal(0,1.5) scale, "
                    "noise 0.5, 0.1% of coordinates boosted 20x"),
    "gpt2s": Workload(
        "gpt2s", d=124_439_808, N=8, grad_dtype="f32", steps=20, eta=0.1, mu=0.001, n=768, r=4,
        data_seed=1003, sketch_seed=2003, family=0, noise=0.3, scale_sigma=1.0,
        tensors=gpt2_small_tensors(),
        description="GPT-2 small layout (148 tensors), per-tensor LogNormal(0,1), noise 0.3"),
    "llama1b": Workload(
        "llama1b", d=1_100_048_384, N=4, grad_dtype="bf16", steps=10, eta=0.05, mu=0.01, n=2048,
        r=4, data_seed=1004, sketch_seed=2004, family=1, scale_sigma=1.0, corr=0.7,
        tensors=tinyllama_tensors(),
        description="TinyLlama-1.1B layout (201 tensors), Student-t(3), per-tensor "
                    "LogNormal(0,1), cross-worker correlation 0.7, bf16"),
    "llama7b": Workload(
        "llama7b", d=6_738_415_616, N=2, grad_dtype="bf16", steps=4, eta=0.05, mu=0.01, n=4096,
        r=4, data_seed=1005, sketch_seed=2005, family=1, scale_sigma=1.0, corr=0.7,
        tensors=llama7b_tensors(), buckets_from_tensors=True,
        description="Llama-7B layout, 35 buckets (embedding, 32 blocks, lm_head: 1% each; "
                    "65 norm rows dense), Student-t(3), LogNormal(0,1), corr 0.7, bf16"),
}

# Per-tensor variants: the same gradients, each tensor compressed in its own
# 2-D view with its own K (1-D tensors whole).
for _base, _views in (("resnet18", resnet18_views()), ("gpt2s", gpt2_small_views()),
                      ("llama1b", tinyllama_views())):
    _w = WORKLOADS[_base]
    WORKLOADS[_base + "_tensors"] = replace(
        _w, name=_base + "_tensors", n=0, views=_views,
        description=_w.description + "; per-tensor views, K = ceil(mu*rows) per matrix, "
                                     "1-D tensors whole")

ORDER = ["tiny", "resnet18", "gpt2s", "llama1b", "llama7b"]
ORDER_TENSORS = ["resnet18_tensors", "gpt2s_tensors", "llama1b_tensors"]


def _check_layouts():
    want = {"resnet18": (62, 11_689_512), "gpt2s": (148, 124_439_808),
            "llama1b": (201, 1_100_048_384), "llama7b": (32 * 7 + 2 + 65, 6_738_415_616)}
    for name, (count, d) in want.items():
        w = WORKLOADS[name]
        assert len(w.tensors) == count and sum(w.tensors) == d == w.d, name
    for name in ORDER_TENSORS:
        w = WORKLOADS[name]
        assert [r * c for r, c in w.views] == w.tensors, name


_check_layouts()
