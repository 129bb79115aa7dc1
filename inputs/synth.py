"""Seeded synthetic workloads for the compressed MoE layer.

Every stream is drawn from ``numpy.random.SeedSequence(MASTER_SEED,
spawn_key=key)`` with a key that names what is drawn (workload, layer, expert,
projection), so any single tensor can be regenerated on its own.

Workloads (shapes follow DeepSeek-V3: hidden 7168, expert intermediate 2048,
256 routed experts in 8 groups, 4 groups and 8 experts per token, routed
scaling 2.5; 192 kept experts is the paper's retention ratio r = 0.75):

* ``tiny``        hidden 512, intermediate 256, 16 experts with 12 kept,
                  1 shared, 2 groups / 1 group / top-2, 8 tokens, all 4-bit;
* ``v3_decode``   V3 shape, 192 of 256 kept, 1 shared; routed gate/up 3-bit,
                  routed down 4-bit, shared 4-bit; 1 and 16 tokens;
* ``v3_prefill``  V3 shape, 2048 tokens, Zipf(1.1)-skewed routing, every
                  tensor's width drawn from {2, 3, 4} with p = (0.6, 0.2, 0.2);
* ``v3_stack``    58 independent V3-shape layers, widths from {2, 3, 4} with
                  p = (0.7, 0.1, 0.2), batch 1, independent inputs per layer;
* ``v3_sweep``    kept in {256, 192, 128} x widths {uniform 2, uniform 4,
                  mixed} x batch {1, 16, 64} x routing {normal, Zipf}.

Value distributions: weights N(0, 0.02) (then quantized by whoever consumes
them), activations N(0, 1) rounded to bfloat16, router logits N(0, 1) in
float32, or ``log p + Gumbel(0, 1)`` with ``p`` a Zipf(1.1) law over a seeded
permutation of the kept experts.
"""
import dataclasses
import zlib

import numpy as np

MASTER_SEED = 20250930
PROJ_GATE, PROJ_UP, PROJ_DOWN = 0, 1, 2


@dataclasses.dataclass(frozen=True)
class LayerShape:
    hidden: int
    inter: int
    n_experts: int
    n_kept: int
    n_shared: int
    n_group: int
    topk_group: int
    top_k: int
    group_topn: int = 2
    norm_topk: int = 1
    routed_scale: float = 2.5
    regroup: int = 0      # 1: routing groups formed over the kept experts only

    def rows_cols(self, proj):
        """(rows, K) of a projection: gate/up are [inter, hidden], down [hidden, inter]."""
        return (self.hidden, self.inter) if proj == PROJ_DOWN else (self.inter, self.hidden)


TINY = LayerShape(hidden=512, inter=256, n_experts=16, n_kept=12, n_shared=1,
                  n_group=2, topk_group=1, top_k=2)
V3 = LayerShape(hidden=7168, inter=2048, n_experts=256, n_kept=192, n_shared=1,
                n_group=8, topk_group=4, top_k=8)

WORKLOADS = {
    "tiny": dict(shape=TINY, tokens=(8,), bits="all4", routing="normal"),
    "v3_decode": dict(shape=V3, tokens=(1, 16), bits="gu3_d4_sh4", routing="normal"),
    "v3_prefill": dict(shape=V3, tokens=(2048,), bits="p234_602020", routing="zipf"),
    "v3_stack": dict(shape=V3, tokens=(1,), bits="p234_701020", routing="normal", layers=58),
    "v3_sweep": dict(shape=V3, tokens=(1, 16, 64), bits=("all2", "all4", "mixed"),
                     routing=("normal", "zipf"), kept=(256, 192, 128)),
}


def _key_int(part):
    if isinstance(part, (int, np.integer)):
        return int(part)
    return zlib.crc32(str(part).encode())


def rng(*key):
    """A numpy Generator for the stream named by ``key`` (strings and ints)."""
    ss = np.random.SeedSequence(MASTER_SEED, spawn_key=tuple(_key_int(k) for k in key))
    return np.random.Generator(np.random.PCG64(ss))


def seed_int(*key):
    """A 63-bit integer seed for the stream named by ``key`` (for torch generators)."""
    ss = np.random.SeedSequence(MASTER_SEED, spawn_key=tuple(_key_int(k) for k in key))
    return int(ss.generate_state(2, np.uint64)[0] >> np.uint64(1))


def expert_mask(shape, *key):
    """uint8 ``[E]``: ``n_kept`` experts kept (1), chosen uniformly at random."""
    r = rng("mask", *key)
    mask = np.zeros(shape.n_experts, np.uint8)
    mask[r.choice(shape.n_experts, shape.n_kept, replace=False)] = 1
    return mask


def bit_plan(shape, plan, *key):
    """Per-tensor widths: (routed int32 ``[E, 3]``, shared int32 ``[n_shared, 3]``).

    Plans: ``all2``/``all4``/``all3``/``all5``/``all6``/``all8``;
    ``gu3_d4_sh<b>`` (routed gate/up 3, routed down 4, shared experts b bits,
    e.g. 6 or 8 for the upgraded shared expert); ``p234_<pppppp>`` (each
    tensor drawn from {2,3,4} with the given percentages); ``wide_all`` (each
    tensor drawn uniformly from {2,3,4,5,6,8}); ``mixed`` (shared 4-bit,
    routed 2-bit)."""
    E, S = shape.n_experts, shape.n_shared
    if plan.startswith("all"):
        b = int(plan[3:])
        return np.full((E, 3), b, np.int32), np.full((S, 3), b, np.int32)
    if plan.startswith("gu3_d4_sh"):
        routed = np.tile(np.array([3, 3, 4], np.int32), (E, 1))
        return routed, np.full((S, 3), int(plan[len("gu3_d4_sh"):]), np.int32)
    if plan == "wide_all":
        r = rng("bits", plan, *key)
        widths = np.array([2, 3, 4, 5, 6, 8], np.int32)
        return r.choice(widths, size=(E, 3)).astype(np.int32), r.choice(widths, size=(S, 3)).astype(np.int32)
    if plan == "mixed":
        return np.full((E, 3), 2, np.int32), np.full((S, 3), 4, np.int32)
    if plan.startswith("p234_"):
        pct = plan[5:]
        p = np.array([int(pct[0:2]), int(pct[2:4]), int(pct[4:6])], np.float64) / 100.0
        r = rng("bits", plan, *key)
        routed = r.choice(np.array([2, 3, 4], np.int32), size=(E, 3), p=p).astype(np.int32)
        shared = r.choice(np.array([2, 3, 4], np.int32), size=(S, 3), p=p).astype(np.int32)
        return routed, shared
    raise ValueError(f"unknown bit plan {plan!r}")


def normal_weights(rows, K, *key, std=0.02):
    """float32 ``[rows, K]`` drawn from N(0, std)."""
    return (rng("w", *key).standard_normal((rows, K), dtype=np.float32) * np.float32(std))


def random_packed(rows, K, bits, *key):
    """A random tensor already in the packed layout: (codes uint8 ``[rows, K*bits/8]``,
    scales uint16 ``[rows, K/32]``).

    Every byte string is a valid packing, so codes are uniform random bytes.
    Scales are binary16 values spread over [0.5, 1.5) times the typical scale
    of N(0, 0.02) weights at this width (about 0.06 / (2**(bits-1) - 1))."""
    r = rng("packed", *key)
    codes = r.integers(0, 256, size=(rows, K * bits // 8), dtype=np.uint8)
    typical = 0.06 / max(1, (1 << (bits - 1)) - 1)
    scales = (r.uniform(0.5, 1.5, size=(rows, K // 32)) * typical).astype(np.float16)
    return codes, scales.view(np.uint16)


def device_random_packed(torch, rows, K, bits, *key, device="cuda"):
    """``random_packed``'s distribution drawn on a GPU with torch's seeded
    generator, for layers too large to draw on the host (the 58-layer stack,
    the pruning/precision sweep): (codes uint8 ``[rows, K*bits/8]``, scales as
    int16 binary16 bit patterns ``[rows, K/32]``), both device tensors.  The
    same key gives the same tensor on every run, so a test can regenerate any
    single tensor and copy it to the host."""
    gen = torch.Generator(device=device)
    gen.manual_seed(seed_int("packed-dev", *key))
    codes = torch.randint(0, 256, (rows, K * bits // 8), generator=gen, device=device, dtype=torch.uint8)
    typical = 0.06 / max(1, (1 << (bits - 1)) - 1)
    u = torch.rand((rows, K // 32), generator=gen, device=device, dtype=torch.float32)
    scales = ((0.5 + u) * typical).to(torch.float16).view(torch.int16)
    return codes, scales


def bf16_from_f32(a):
    """Round float32 to the nearest bfloat16 (ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def activations(n, H, *key):
    """bfloat16 bit patterns ``[n, H]`` of N(0, 1) draws."""
    return bf16_from_f32(rng("x", *key).standard_normal((n, H), dtype=np.float32))


def router_weight(E, H, *key):
    """float32 gate ``[E, H]`` of N(0, 1/H) draws: with N(0, 1) activations the
    logits are about N(0, 1)."""
    return (rng("router_w", *key).standard_normal((E, H), dtype=np.float32)
            / np.float32(np.sqrt(H))).astype(np.float32)


def grid_activations(n, H, *key):
    """bfloat16 bit patterns ``[n, H]`` of integers drawn uniformly from -4..4."""
    return bf16_from_f32(rng("xgrid", *key).integers(-4, 5, size=(n, H)).astype(np.float32))


def grid_router_weight(E, H, *key):
    """float32 gate ``[E, H]``: integers from -64..64 times 2^-12.  Against
    ``grid_activations`` every product and every partial sum of a row of up to
    8192 terms is a multiple of 2^-12 below 2^12 in magnitude, so float32
    arithmetic computes the logits exactly in any order."""
    ints = rng("wgrid", *key).integers(-64, 65, size=(E, H)).astype(np.float32)
    return (ints * np.float32(2.0 ** -12)).astype(np.float32)


def normal_logits(n, E, *key):
    """float32 ``[n, E]`` router logits drawn from N(0, 1)."""
    return rng("logits", *key).standard_normal((n, E), dtype=np.float32)


def zipf_logits(n, mask, *key, s=1.1):
    """float32 ``[n, E]``: ``log p_{pi(e)} + Gumbel(0, 1)`` for kept experts.

    ``p`` is Zipf(s) over the kept experts under a seeded permutation ``pi``,
    so the Gumbel-max top-k draws experts without replacement in proportion to
    ``p``.  Pruned experts get the most popular expert's law, so the router's
    masking is exercised."""
    mask = np.asarray(mask).astype(bool)
    E = mask.shape[0]
    r = rng("zipf", *key)
    kept = np.nonzero(mask)[0]
    ranks = np.empty(E, np.float64)
    ranks[kept] = r.permutation(len(kept)) + 1.0
    ranks[~mask] = 1.0
    logp = -s * np.log(ranks)
    logp -= np.log(np.sum(np.arange(1, len(kept) + 1, dtype=np.float64) ** -s))
    gumbel = r.gumbel(0.0, 1.0, size=(n, E))
    return (logp[None, :] + gumbel).astype(np.float32)


# ---------------------------------------------------------------------------
# Model-level inventory for the bit-allocation planner.
def v3_tensor_inventory(n_kept=192):
    """The quantizable matrices of a DeepSeek-V3-architecture model (61 layers,
    the first 3 dense, 58 MoE; multi-head latent attention with q rank 1536,
    kv rank 512, 128 heads of 128 + 64 rope dims; dense intermediate 18432;
    one shared and ``n_kept`` routed experts of intermediate 2048; vocabulary
    129280), one entry per matrix, routed experts as one tensor per layer and
    projection.  Norm vectors are left out.

    Returns (names, params, kind, layer, layer_params): kind 0 = other,
    1/2/3 = routed gate/up/down; layer = MoE layer position (0..57) of routed
    tensors, else -1; layer_params = parameters of the tensor's layer (the
    tensor itself for the embedding and output matrices)."""
    H, vocab, heads = 7168, 129280, 128
    attn = {"attn_q_a": H * 1536, "attn_q_b": 1536 * heads * 192, "attn_kv_a_mqa": H * 576,
            "attn_kv_b": 512 * heads * 256, "attn_output": heads * 128 * H}
    names, params, kind, layer, owner = [], [], [], [], []

    def add(name, p, k=0, pos=-1, lid=None):
        names.append(name)
        params.append(int(p))
        kind.append(k)
        layer.append(pos)
        owner.append(lid)
    add("token_embd", vocab * H, lid="token_embd")
    for L in range(61):
        for a, p in attn.items():
            add(f"blk.{L}.{a}", p, lid=L)
        if L < 3:
            for f in ("ffn_gate", "ffn_up", "ffn_down"):
                add(f"blk.{L}.{f}", H * 18432, lid=L)
            continue
        pos = L - 3
        add(f"blk.{L}.ffn_gate_inp", 256 * H, lid=L)
        for f in ("ffn_gate_shexp", "ffn_up_shexp", "ffn_down_shexp"):
            add(f"blk.{L}.{f}", H * 2048, lid=L)
        for k, f in ((1, "ffn_gate_exps"), (2, "ffn_up_exps"), (3, "ffn_down_exps")):
            add(f"blk.{L}.{f}", n_kept * H * 2048, k, pos, lid=L)
    add("output", vocab * H, lid="output")
    totals = {}
    for p, o in zip(params, owner):
        totals[o] = totals.get(o, 0) + p
    layer_params = [totals[o] for o in owner]
    return names, params, kind, layer, layer_params


def synthetic_perplexities(params, layer_params, *key, ppl_low=12.0):
    """Seeded stand-ins for PPL(Q_low) and PPL(Q_high, t): raising tensor t
    lowers the perplexity by rho_t * 0.05 * LogNormal(0, 1)."""
    r = rng("ppl", *key)
    rho = np.asarray(params, np.float64) / np.asarray(layer_params, np.float64)
    drop = rho * 0.05 * np.exp(r.standard_normal(len(params)))
    return float(ppl_low), (ppl_low - drop).astype(np.float64)
