"""Shapes and seeded values of one rank's training-state shard.

A rank's protected state in the paper is its optimizer-state shard plus its
model-parameter shard (Sec. V-B, D2H paragraph).  Here each parameter tensor
contributes four fragments, in this order: the bf16 parameter, its fp32
master copy and the fp32 Adam moments m and v (14 bytes per parameter).
Values: master ~ N(0, 0.02^2), parameter = bf16(master) (round to nearest
even), m ~ N(0, 1e-3^2), v = (N(0, 1e-3^2))^2; every fragment draws from its
own generator seeded from (1000 + workload id, fragment index).

Workloads (ids 1-6):
  1  4-layer GPT, hidden 512, FFN 2048, vocab 8192, 512 positions (17.07M params), 4 MiB chunks
  2  24-layer GPT, hidden 2048, FFN 8192, vocab 50304, 2048 positions (1.316B params), 64 MiB chunks
  3  one rank of a 65B LLaMA under TP=8 x PP=8: 10 layers, hidden 8192, FFN 22016/8 (1.012B params)
  4  7B LLaMA: 32 layers, hidden 4096, FFN 11008, vocab 32000 (6.738B params)
  5  4096 fragments, log-uniform sizes rescaled to 8 GiB in total, bf16/fp32 alternating
  6  workload 3 in full precision, the paper's training setting (Sec. VII): the parameter is fp32 too
     (equal to its master copy), 16 bytes per parameter
"""
import math

import numpy as np

# dtype tags carried in the fragment table (the library treats bytes as opaque)
DT_BYTES, DT_BF16, DT_FP32 = 0, 1, 2
# class tags: what part of the rank state a fragment is
CLS_PARAM, CLS_MASTER, CLS_ADAM_M, CLS_ADAM_V = 0, 1, 2, 3
CLASS_DTYPE = {CLS_PARAM: DT_BF16, CLS_MASTER: DT_FP32, CLS_ADAM_M: DT_FP32, CLS_ADAM_V: DT_FP32}
ELEM_BYTES = {DT_BYTES: 1, DT_BF16: 2, DT_FP32: 4}

MiB = 1 << 20
GiB = 1 << 30

WORKLOADS = {
    1: dict(name="gpt-tiny-4L-h512", kind="gpt", layers=4, hidden=512, ffn=2048, vocab=8192, seq=512,
            chunk=4 * MiB),
    2: dict(name="gpt-1.3B-24L-h2048", kind="gpt", layers=24, hidden=2048, ffn=8192, vocab=50304, seq=2048,
            chunk=64 * MiB),
    3: dict(name="llama65B-tp8pp8-rank-10L-h8192", kind="llama", layers=10, hidden=8192, ffn=22016, vocab=32000,
            tp=8, embed=False, head=False, chunk=64 * MiB),
    4: dict(name="llama-7B-32L-h4096", kind="llama", layers=32, hidden=4096, ffn=11008, vocab=32000, tp=1,
            embed=True, head=True, chunk=64 * MiB),
    5: dict(name="stress-4096-frag-8GiB", kind="stress", n=4096, total=8 * GiB, lo=1024, hi=64 * MiB,
            chunk=64 * MiB),
    6: dict(name="llama65B-tp8pp8-rank-10L-h8192-fp32", kind="llama", layers=10, hidden=8192, ffn=22016,
            vocab=32000, tp=8, embed=False, head=False, chunk=64 * MiB, fp32=True),
}

# bf16 GEMM that stands in for forward/backward compute in the overlap runs
OVERLAP_GEMM = {3: (8192, 8192, 2752), 4: (8192, 4096, 11008), 6: (8192, 8192, 2752)}


def gpt_param_shapes(layers, hidden, ffn, vocab, seq):
    h = hidden
    shapes = [("wte", (vocab, h)), ("wpe", (seq, h))]
    for l in range(layers):
        p = "h%d." % l
        shapes += [(p + "ln1.w", (h,)), (p + "ln1.b", (h,)),
                   (p + "attn.qkv.w", (3 * h, h)), (p + "attn.qkv.b", (3 * h,)),
                   (p + "attn.proj.w", (h, h)), (p + "attn.proj.b", (h,)),
                   (p + "ln2.w", (h,)), (p + "ln2.b", (h,)),
                   (p + "mlp.fc1.w", (ffn, h)), (p + "mlp.fc1.b", (ffn,)),
                   (p + "mlp.fc2.w", (h, ffn)), (p + "mlp.fc2.b", (h,))]
    shapes += [("ln_f.w", (h,)), ("ln_f.b", (h,))]
    return shapes


def llama_param_shapes(layers, hidden, ffn, vocab, tp=1, embed=True, head=True):
    h = hidden
    f = ffn // tp
    shapes = []
    if embed:
        shapes.append(("embed", (vocab, h)))
    for l in range(layers):
        p = "layers.%d." % l
        shapes += [(p + "attn_norm", (h,)),
                   (p + "q", (h // tp, h)), (p + "k", (h // tp, h)), (p + "v", (h // tp, h)), (p + "o", (h, h // tp)),
                   (p + "ffn_norm", (h,)),
                   (p + "gate", (f, h)), (p + "up", (f, h)), (p + "down", (h, f))]
    if head:
        shapes += [("norm", (h,)), ("lm_head", (vocab, h))]
    return shapes


def param_shapes(wid):
    w = WORKLOADS[wid]
    if w["kind"] == "gpt":
        return gpt_param_shapes(w["layers"], w["hidden"], w["ffn"], w["vocab"], w["seq"])
    if w["kind"] == "llama":
        return llama_param_shapes(w["layers"], w["hidden"], w["ffn"], w["vocab"], w["tp"], w["embed"], w["head"])
    raise ValueError("workload %d has no parameter shapes" % wid)


def n_params(wid):
    return sum(math.prod(s) for _, s in param_shapes(wid))


def stress_sizes(n=4096, total=8 * GiB, lo=1024, hi=64 * MiB, seed=1005):
    """Fragment byte sizes of the restore stress workload.  The stated range
    (log-uniform on [1 KiB, 64 MiB]) and total (8 GiB) disagree, so the draws
    are rescaled to the total: sizes are drawn log-uniform, scaled by
    total/sum, rounded down to the element size (bf16 at even indices, fp32 at
    odd ones), floored at 1 KiB, and the residual goes to the largest
    fragment.  Returns (sizes, dtype tags)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    raw = np.exp(rng.uniform(math.log(lo), math.log(hi), n))
    scaled = raw * (total / raw.sum())
    dts = [DT_BF16 if i % 2 == 0 else DT_FP32 for i in range(n)]
    sizes = []
    for x, dt in zip(scaled, dts):
        e = ELEM_BYTES[dt]
        s = max(int(x) // e * e, lo)
        sizes.append(s)
    big = int(np.argmax(sizes))
    resid = total - sum(sizes)
    e = ELEM_BYTES[dts[big]]
    if resid % e:
        # move the odd 2 bytes onto the first bf16 fragment
        sizes[0] += resid % e
        resid -= resid % e
    sizes[big] += resid
    assert sum(sizes) == total and min(sizes) >= lo
    return sizes, dts


def fragment_plan(wid):
    """[(name, nbytes, dtype tag, class tag)] in registration order."""
    if WORKLOADS[wid]["kind"] == "stress":
        w = WORKLOADS[wid]
        sizes, dts = stress_sizes(w["n"], w["total"], w["lo"], w["hi"])
        return [("frag%d" % i, s, dt, CLS_MASTER if dt == DT_FP32 else CLS_PARAM)
                for i, (s, dt) in enumerate(zip(sizes, dts))]
    plan = []
    fp32 = WORKLOADS[wid].get("fp32", False)
    for name, shape in param_shapes(wid):
        numel = math.prod(shape)
        for cls, suffix in [(CLS_PARAM, ""), (CLS_MASTER, ".master"), (CLS_ADAM_M, ".exp_avg"),
                            (CLS_ADAM_V, ".exp_avg_sq")]:
            dt = DT_FP32 if fp32 else CLASS_DTYPE[cls]
            plan.append((name + suffix, numel * ELEM_BYTES[dt], dt, cls))
    return plan


def payload_bytes(wid):
    return sum(p[1] for p in fragment_plan(wid))


def fragment_seed(wid, index):
    return ((1000 + wid) << 24) | index


def make_state(wid, device="cuda"):
    """Allocate and fill the shard's fragments as separate torch tensors.
    Returns (tensors, plan).  Parameter-major order: param, master, m, v."""
    import torch

    plan = fragment_plan(wid)
    out = []
    if WORKLOADS[wid]["kind"] == "stress":
        for i, (_, nb, dt, _) in enumerate(plan):
            g = torch.Generator(device=device).manual_seed(fragment_seed(wid, i))
            if dt == DT_BF16:
                t = (torch.randn(nb // 2, generator=g, device=device) * 0.02).to(torch.bfloat16)
            else:
                t = torch.randn(nb // 4, generator=g, device=device) * 1e-3
            out.append(t)
        return out, plan
    for i in range(0, len(plan), 4):
        numel = plan[i][1] // ELEM_BYTES[plan[i][2]]
        g = torch.Generator(device=device).manual_seed(fragment_seed(wid, i))
        master = torch.randn(numel, generator=g, device=device) * 0.02
        param = master.clone() if plan[i][2] == DT_FP32 else master.to(torch.bfloat16)
        g = torch.Generator(device=device).manual_seed(fragment_seed(wid, i + 2))
        m = torch.randn(numel, generator=g, device=device) * 1e-3
        g = torch.Generator(device=device).manual_seed(fragment_seed(wid, i + 3))
        v = torch.randn(numel, generator=g, device=device) * 1e-3
        v.mul_(v)
        out += [param, master, m, v]
    return out, plan


def adversarial_fragments(device="cuda"):
    """Fragments whose raw bits a float path would alter: NaN payloads, -0,
    subnormals, +-Inf and all-ones words, in bf16, fp32 and raw bytes, with
    ragged lengths."""
    import torch

    f32_bits = [0x7FC00001, 0xFFFFFFFF, 0x80000000, 0x00000001, 0x7F800000, 0xFF800000, 0x7F800001,
                0x807FFFFF, 0x00000000, 0x3F800000]
    bf16_bits = [0x7FC1, 0xFFFF, 0x8000, 0x0001, 0x7F80, 0xFF80, 0x7F81, 0x807F]
    a = torch.tensor(f32_bits * 37, dtype=torch.int64).to(torch.int32).view(torch.float32)
    b = torch.tensor(bf16_bits * 101, dtype=torch.int32).to(torch.int16).view(torch.bfloat16)
    c = torch.full((4099,), 0xFF, dtype=torch.uint8)
    d = torch.tensor([0x80, 0x00, 0xFF, 0x01, 0x7F] * 13, dtype=torch.uint8)
    return [t.to(device) for t in (a, b, c, d)]


def misaligned_views(device="cuda", seed=7):
    """Slices of flat buffers at odd element and byte offsets, as a
    distributed optimizer's flat buffers hand out."""
    import torch

    g = torch.Generator(device="cpu").manual_seed(seed)
    flat16 = torch.randint(-32768, 32767, (300_000,), generator=g, dtype=torch.int16).view(torch.bfloat16)
    flat32 = torch.randn(200_000, generator=g)
    flat8 = torch.randint(0, 256, (100_000,), generator=g, dtype=torch.uint8)
    flat16, flat32, flat8 = flat16.to(device), flat32.to(device), flat8.to(device)
    views = [flat16[1:1001], flat16[1003:70_000], flat16[70_001:70_002], flat16[70_005:250_017],
             flat32[1:5], flat32[7:150_003], flat8[3:4000], flat8[4001:4002], flat8[4007:99_999],
             flat16[250_019:299_999]]
    return views, (flat16, flat32, flat8)


def flip_positions(chunk_ranges, n_flips=32, seed=2005, distinct_chunks=True):
    """Seeded single-bit flip positions for the integrity test: n_flips
    distinct chunks, and in each a uniform 8-byte word of the chunk and a
    uniform bit 0-63.  chunk_ranges is [(lo, hi)] of image bytes.  Returns
    [(chunk, byte offset in the image, bit 0-7 within that byte)]."""
    rng = np.random.Generator(np.random.PCG64(seed))
    nc = len(chunk_ranges)
    if distinct_chunks:
        chunks = sorted(int(c) for c in rng.choice(nc, size=min(n_flips, nc), replace=False))
    else:
        chunks = sorted(int(c) for c in rng.integers(0, nc, n_flips))
    out = []
    for c in chunks:
        lo, hi = chunk_ranges[c]
        word = int(rng.integers(0, (hi - lo) // 8))
        bit = int(rng.integers(0, 64))
        out.append((c, lo + 8 * word + bit // 8, bit % 8))
    return out
