"""The five LM-GC workloads: decoder shapes, serialisation and value distributions.

Decoder shapes follow the LLMs the paper uses as priors (Section 5.1: TinyLlama
1.1B and LLaMA-2 7B; the GPT-2-small shape and a tiny fp32 decoder are extra
test shapes).  Window sizes follow the paper's window ablation (Fig. 2 caption:
256 ... 4096 tokens).  Weights are random-init, because no checkpoint is
available; every matrix and embedding is N(0, 0.02), norm gains are 1 and
biases are 0.

Serialisation (Section 4, "Serialization"): every float32 becomes 8 hex digits
(one per 4-bit partition) followed by one separator token; the tokenizer is a
fixed one-id-per-character map (lowercase ASCII codes for the digits, 32 for
the space separator of the H_s variant).
"""
from dataclasses import dataclass, field, replace
from typing import List, Tuple

HEX_CHARS = "0123456789abcdef"


@dataclass(frozen=True)
class ModelShape:
    arch: str            # "llama" (RMSNorm, RoPE, SwiGLU, untied head) | "gpt2"
    dtype: str           # "f32" | "bf16"
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    d_ff: int
    vocab: int
    max_pos: int
    rope_theta: float = 10000.0
    norm_eps: float = 1e-5

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads


@dataclass(frozen=True)
class SerialSpec:
    bytes_per_value: int          # 4 (float32) | 2 | 1 (8-bit indices)
    bytes_per_group: int          # separator after every this many bytes; 0 = none
    msb_first: int                # 1: most significant byte/nibble first
    window: int                   # LM context window W (tokens)
    bos_id: int
    pad_id: int
    sep_id: int
    hex_ids: Tuple[int, ...] = field(default=tuple(ord(c) for c in HEX_CHARS))
    sep2_id: int = -1             # second separator token after each group; -1 = none
    renorm: int = 0               # 1: tables renormalised over the alphabet (no escape mass)


# The separators of the paper's hexadecimal serialisations (Section 5.2,
# Table 1), as (sep_id, sep2_id) character codes; H_n is bytes_per_group = 0.
SEPARATORS = {"H_s": (ord(" "), -1), "H_c": (ord(","), -1), "H_semi": (ord(";"), -1),
              "H_c+s": (ord(","), ord(" "))}


def hex_serial(window: int, bos_id: int, bytes_per_value: int = 4,
               bytes_per_group: int = None, msb_first: int = 1,
               sep_id: int = 32, sep2_id: int = -1) -> SerialSpec:
    """Hexadecimal serialisation (H_s by default: a space after each group)."""
    if bytes_per_group is None:
        bytes_per_group = bytes_per_value
    return SerialSpec(bytes_per_value=bytes_per_value,
                      bytes_per_group=bytes_per_group, msb_first=msb_first,
                      window=window, bos_id=bos_id, pad_id=bos_id,
                      sep_id=sep_id, sep2_id=sep2_id)


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    serial: SerialSpec
    n_values: int
    dist: str                     # see gen.gen_values
    batch: int                    # windows per lmgc_probs call
    value_seed: int = 0
    weight_seed: int = 1
    lossy: str = ""               # lossy steps applied before LM-GC; see parse_lossy

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


M = 1 << 20

TINY = Workload(
    name="tiny",
    model=ModelShape(arch="llama", dtype="f32", n_layers=2, d_model=128,
                     n_heads=4, n_kv_heads=4, d_ff=512, vocab=256, max_pos=256),
    serial=hex_serial(window=256, bos_id=1),
    n_values=4096, dist="normal:1e-3", batch=144)

GPT2 = Workload(
    name="gpt2",
    model=ModelShape(arch="gpt2", dtype="bf16", n_layers=12, d_model=768,
                     n_heads=12, n_kv_heads=12, d_ff=3072, vocab=50257,
                     max_pos=1024),
    serial=hex_serial(window=1024, bos_id=50256),
    n_values=1 * M, dist="laplace:5e-4", batch=32)

TINYLLAMA = Workload(
    name="tinyllama",
    model=ModelShape(arch="llama", dtype="bf16", n_layers=22, d_model=2048,
                     n_heads=32, n_kv_heads=4, d_ff=5632, vocab=32000,
                     max_pos=2048),
    serial=hex_serial(window=2048, bos_id=1),
    n_values=4 * M, dist="mixture:1e-4:0.01:1e-2", batch=16)

LLAMA7B = Workload(
    name="7b",
    model=ModelShape(arch="llama", dtype="bf16", n_layers=32, d_model=4096,
                     n_heads=32, n_kv_heads=32, d_ff=11008, vocab=32000,
                     max_pos=4096),
    serial=hex_serial(window=4096, bos_id=1),
    n_values=2 * M, dist="laplace:1e-3", batch=8)

LOSSY7B = Workload(
    name="lossy7b",
    model=LLAMA7B.model,
    serial=hex_serial(window=4096, bos_id=1, bytes_per_value=1),
    n_values=8 * M, dist="normal:1e-3", batch=8, lossy="sparsify:10+quantize:8")

WORKLOADS = {w.name: w for w in (TINY, GPT2, TINYLLAMA, LLAMA7B, LOSSY7B)}


# ----------------------------------------------------------- lossy steps --
# The lossy schemes LM-GC is composed with (Section 5.4), as a '+'-joined
# list applied left to right:
#   sparsify:<percent>   keep that percentage of the values (float32 stream)
#   quantize:<bits>      linear quantisation to <bits>-bit indices (Eq. 4);
#                        1..8 bits give a uint8 stream, 9..16 a uint16 stream
#   sign                 one sign bit per value, eight to a byte (SignSGD)
LOSSY_VARIANTS = {
    "q16": "quantize:16", "q8": "quantize:8", "sign": "sign",
    "s50": "sparsify:50", "s25": "sparsify:25", "s10": "sparsify:10",
    "s10q8": "sparsify:10+quantize:8",
}


def parse_lossy(spec: str) -> List[Tuple[str, int]]:
    """'sparsify:10+quantize:8' -> [('sparsify', 10), ('quantize', 8)]."""
    steps: List[Tuple[str, int]] = []
    for part in filter(None, spec.split("+")):
        name, _, arg = part.partition(":")
        if name == "sparsify" and arg and 0 <= int(arg) <= 100:
            steps.append((name, int(arg)))
        elif name == "quantize" and arg and 1 <= int(arg) <= 16:
            steps.append((name, int(arg)))
        elif name == "sign" and not arg:
            steps.append((name, 0))
        else:
            raise ValueError(f"bad lossy step {part!r}")
    kinds = [k for k, _ in steps]
    if ("sign" in kinds or "quantize" in kinds) and kinds[-1] not in ("sign", "quantize"):
        raise ValueError("quantize/sign must be the last lossy step")
    if kinds.count("sign") + kinds.count("quantize") > 1:
        raise ValueError("at most one of quantize/sign")
    return steps


def lossy_bytes_per_value(spec: str) -> int:
    """Bytes per element of the stream a lossy spec produces."""
    steps = parse_lossy(spec)
    if not steps or steps[-1][0] == "sparsify":
        return 4
    if steps[-1][0] == "sign":
        return 1
    return 1 if steps[-1][1] <= 8 else 2


def get_workload(name: str) -> Workload:
    try:
        return WORKLOADS[name]
    except KeyError:
        raise KeyError(f"unknown workload {name!r}; have {sorted(WORKLOADS)}")
