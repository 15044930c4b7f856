"""Workload shapes of the partition path, after the paper's model families
(Llama-2 and Falcon, Experimentation section) at their published
architecture sizes, and the partition rule of Eq. 1.

A workload fixes: the rank's partition length n (total parameters / P,
the ZeRO-3 partition), the layer that is gathered (N elements over P'
node-local secondary shards of s elements each), the quantization block and
the Adam hyperparameters.
"""
from dataclasses import dataclass

BLOCK = 256


def secondary_elems(layer_elems, secondary_world, block=BLOCK):
    """Elements of one secondary shard: |L|/P' (Eq. 1), rounded up to whole
    quantization blocks so that blocks never straddle shards; the last shard
    is zero-padded."""
    per = (layer_elems + secondary_world - 1) // secondary_world
    return (per + block - 1) // block * block


def llama2_layer(hidden, mlp):
    # q, k, v, o projections; gate, up, down; two RMSNorm weights
    return 4 * hidden * hidden + 3 * hidden * mlp + 2 * hidden


def llama2_total(hidden, mlp, layers, vocab):
    # untied embedding and LM head, final norm
    return layers * llama2_layer(hidden, mlp) + 2 * vocab * hidden + hidden


def falcon_layer(hidden, mlp, head_dim, kv_heads, norms):
    # fused qkv (all query heads + kv_heads keys and values), dense, MLP in/out,
    # `norms` LayerNorms with weight and bias
    qkv = hidden * (hidden + 2 * kv_heads * head_dim)
    return qkv + hidden * hidden + 2 * hidden * mlp + 2 * norms * hidden


@dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int            # seed component of every synthetic array of this workload
    n: int                 # rank partition (elements of fp32 master/m/v/grad)
    layer_elems: int       # N of the gathered layer
    secondary_world: int   # P'
    world: int             # P (simulated ranks)
    block: int = BLOCK
    lr: float = 1e-4
    beta1: float = 0.9
    beta2: float = 0.95
    eps: float = 1e-8
    weight_decay: float = 0.1
    iterations: int = 1
    # the backward pass of one step gathers this many layers, one after the
    # other, cycling over `distinct_layers` separately stored synthetic layers
    layers_gathered: int = 1
    distinct_layers: int = 1
    notes: str = ""

    @property
    def shard_elems(self):
        return secondary_elems(self.layer_elems, self.secondary_world, self.block)

    @property
    def adam(self):
        return dict(lr=self.lr, beta1=self.beta1, beta2=self.beta2, eps=self.eps,
                    weight_decay=self.weight_decay)


LLAMA2_7B_TOTAL = llama2_total(4096, 11008, 32, 32000)       # 6,738,415,616
LLAMA2_13B_TOTAL = llama2_total(5120, 13824, 40, 32000)      # 13,015,864,320
FALCON_40B_LAYER = falcon_layer(8192, 32768, 64, 8, 2)      # 679,510,016
# 60 layers + embedding and untied head at vocab 65,024 + final LayerNorm
FALCON_40B_TOTAL = 60 * FALCON_40B_LAYER + 2 * 65024 * 8192 + 2 * 8192

WORKLOADS = {
    "tiny": Workload(
        name="tiny", cfg_id=0, n=1 << 20, layer_elems=4 << 20, secondary_world=2, world=4,
        notes="1,048,576-element rank partition, 4 simulated ranks, P'=2"),
    "falcon-7b-layer": Workload(
        name="falcon-7b-layer", cfg_id=1, n=secondary_elems(falcon_layer(4544, 18176, 64, 1, 1), 8),
        layer_elems=falcon_layer(4544, 18176, 64, 1, 1), secondary_world=8, world=8,
        notes="one Falcon-7B decoder layer gathered from 8 secondary shards"),
    "llama-2-7b": Workload(
        name="llama-2-7b", cfg_id=2, n=LLAMA2_7B_TOTAL // 32, layer_elems=llama2_layer(4096, 11008),
        secondary_world=8, world=32, notes="Llama-2-7B over 32 ranks"),
    "llama-2-13b": Workload(
        name="llama-2-13b", cfg_id=3, n=LLAMA2_13B_TOTAL // 64,
        layer_elems=llama2_layer(5120, 13824), secondary_world=8, world=64,
        notes="Llama-2-13B over 64 ranks; one 5120-hidden layer gathered from 8 shards"),
    "falcon-40b": Workload(
        name="falcon-40b", cfg_id=4, n=FALCON_40B_TOTAL // 128, layer_elems=FALCON_40B_LAYER,
        secondary_world=8, world=128, iterations=10, layers_gathered=60, distinct_layers=2,
        notes="Falcon-40B over 128 ranks, 10 iterations; each step gathers its 60 layers, "
              "cycling over 2 stored layers"),
}

# Algorithmic HBM bytes per element of each kernel (no re-reads, no recompute)
BYTES_ADAM = 30.0                      # read p, m, v, g (16 B); write p, m, v (12 B) + bf16 (2 B)
BYTES_REFRESH = 4.0                    # read 2 B, write 2 B


def bytes_quant(n, block=BLOCK):
    return 2 * n + n + 4 * ((n + block - 1) // block)


def bytes_refresh_quant(n, block=BLOCK):
    # the refresh and its quantization in one pass: read 2 B once, write the
    # secondary (2 B), the codes (1 B) and one fp32 scale per block
    return 2 * n + 2 * n + n + 4 * ((n + block - 1) // block)


def bytes_gather(shard_elems, num_shards, layer_elems, block=BLOCK):
    # reads whole shards only as far as the layer reaches
    read_codes = layer_elems
    blocks = 0
    for j in range(num_shards):
        valid = max(0, min(shard_elems, layer_elems - j * shard_elems))
        blocks += (valid + block - 1) // block
    return read_codes + 4 * blocks + 2 * layer_elems


def bytes_fused(n, block=BLOCK):
    # Adam's 30 B, the secondary copy written (2 B), the codes and scales
    # written (1 B + 4 B per block); the primary is not read back
    return 32 * n + n + 4 * ((n + block - 1) // block)


def bytes_quant_i4(n, block=BLOCK):
    # read fp32 (4 B), write packed int4 (0.5 B) and one fp32 scale per block
    return 4 * n + (n + 1) // 2 + 4 * ((n + block - 1) // block)


def bytes_reduce_i4(n, num_src, block=BLOCK):
    # read every source's packed codes and scales, write the fp32 result
    return num_src * ((n + 1) // 2 + 4 * ((n + block - 1) // block)) + 4 * n


def bytes_receive_adam(n, num_src, block=BLOCK):
    # the partition step without its gradient read (26 B: p, m, v in and out,
    # bf16 out) plus every source's packed codes and scales
    return 26 * n + num_src * ((n + 1) // 2 + 4 * ((n + block - 1) // block))


def bytes_fused_receive(n, num_src, block=BLOCK, grad_block=BLOCK):
    # the receive step's 26 B + sources, the primary read back by nobody: the
    # secondary (2 B), the codes (1 B) and the int8 scales written
    return (bytes_receive_adam(n, num_src, grad_block) + 2 * n + n
            + 4 * ((n + block - 1) // block))
