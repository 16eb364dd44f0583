"""Parameter shape lists of the paper's four workloads, in registration order.

The paper measures ResNet-50, ResNet-152, BERT-Base and BERT-Large
(Section III-A, "Models", and Table 1).  The compressor only sees the
shapes of the gradients, so a workload here is the ordered list of
parameter shapes that a PyTorch model registers (forward order); the
backward order is its reverse.

This module holds workload descriptions only: no eligibility rule, no
reshape and no bucketing (those are the method's arithmetic and live on
each side separately).
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import List, Sequence, Tuple

Shape = Tuple[int, ...]


@dataclass(frozen=True)
class Param:
    name: str
    shape: Shape

    @property
    def numel(self) -> int:
        n = 1
        for d in self.shape:
            n *= d
        return n


def _bn(prefix: str, c: int) -> List[Param]:
    return [Param(prefix + ".weight", (c,)), Param(prefix + ".bias", (c,))]


def resnet(blocks: Sequence[int], num_classes: int = 1000) -> List[Param]:
    """Bottleneck ResNet (expansion 4, stage widths 64/128/256/512), torchvision order.

    ResNet-50 is blocks (3, 4, 6, 3); ResNet-152 is (3, 8, 36, 3).
    """
    ps: List[Param] = [Param("conv1.weight", (64, 3, 7, 7))] + _bn("bn1", 64)
    in_ch = 64
    for stage, (nblk, width) in enumerate(zip(blocks, (64, 128, 256, 512))):
        for b in range(nblk):
            pre = f"layer{stage + 1}.{b}"
            ps.append(Param(pre + ".conv1.weight", (width, in_ch, 1, 1)))
            ps += _bn(pre + ".bn1", width)
            ps.append(Param(pre + ".conv2.weight", (width, width, 3, 3)))
            ps += _bn(pre + ".bn2", width)
            ps.append(Param(pre + ".conv3.weight", (4 * width, width, 1, 1)))
            ps += _bn(pre + ".bn3", 4 * width)
            if b == 0:
                ps.append(Param(pre + ".downsample.0.weight", (4 * width, in_ch, 1, 1)))
                ps += _bn(pre + ".downsample.1", 4 * width)
            in_ch = 4 * width
    ps.append(Param("fc.weight", (num_classes, 512 * 4)))
    ps.append(Param("fc.bias", (num_classes,)))
    return ps


def bert(hidden: int, layers: int, ffn: int, vocab: int = 30522, max_pos: int = 512,
         full: bool = False) -> List[Param]:
    """BERT encoder parameters in HuggingFace registration order.

    ``full=False`` is the encoder-only set of the benchmark workloads: word and
    position embeddings, the embedding LayerNorm and the encoder layers.
    ``full=True`` adds the token-type embedding, the pooler and the
    pre-training heads (masked-LM transform, LayerNorm and decoder bias with the
    decoder weight tied to the word embedding, next-sentence head), which is
    the parameter count Table 1 quotes.
    """
    h = hidden
    ps: List[Param] = [Param("embeddings.word_embeddings.weight", (vocab, h)),
                       Param("embeddings.position_embeddings.weight", (max_pos, h))]
    if full:
        ps.append(Param("embeddings.token_type_embeddings.weight", (2, h)))
    ps += _bn("embeddings.LayerNorm", h)
    for i in range(layers):
        pre = f"encoder.layer.{i}"
        for nm in ("attention.self.query", "attention.self.key", "attention.self.value",
                   "attention.output.dense"):
            ps.append(Param(f"{pre}.{nm}.weight", (h, h)))
            ps.append(Param(f"{pre}.{nm}.bias", (h,)))
        ps += _bn(f"{pre}.attention.output.LayerNorm", h)
        ps.append(Param(f"{pre}.intermediate.dense.weight", (ffn, h)))
        ps.append(Param(f"{pre}.intermediate.dense.bias", (ffn,)))
        ps.append(Param(f"{pre}.output.dense.weight", (h, ffn)))
        ps.append(Param(f"{pre}.output.dense.bias", (h,)))
        ps += _bn(f"{pre}.output.LayerNorm", h)
    if full:
        ps.append(Param("pooler.dense.weight", (h, h)))
        ps.append(Param("pooler.dense.bias", (h,)))
        ps.append(Param("cls.predictions.transform.dense.weight", (h, h)))
        ps.append(Param("cls.predictions.transform.dense.bias", (h,)))
        ps += _bn("cls.predictions.transform.LayerNorm", h)
        ps.append(Param("cls.predictions.bias", (vocab,)))
        ps.append(Param("cls.seq_relationship.weight", (2, h)))
        ps.append(Param("cls.seq_relationship.bias", (2,)))
    return ps


def resnet50() -> List[Param]:
    return resnet((3, 4, 6, 3))


def resnet152() -> List[Param]:
    return resnet((3, 8, 36, 3))


def bert_base(full: bool = False) -> List[Param]:
    return bert(768, 12, 3072, full=full)


def bert_large(full: bool = False) -> List[Param]:
    return bert(1024, 24, 4096, full=full)


def single_conv() -> List[Param]:
    """One 3x3 convolution with 256 output and 64 input channels (a 256 x 576 gradient)."""
    return [Param("conv.weight", (256, 64, 3, 3))]
