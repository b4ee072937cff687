"""Example programs for the front end, written in its text form.

`gpt2_layers` writes GPT-2-shaped decoder layers (Sec. 5: GPT-2 is the
paper's inference example) placed by hand the way Sec. 2.2 describes
distributed programs: each layer's attention heads and MLP columns split
over `tp` devices (Megatron-style: QKV and fc1 column-parallel, the output
projection and fc2 row-parallel, each followed by an AllReduce), layers
grouped into `pp` pipeline stages joined by Sends.  The input is flattened
from (batch, seq, d) to (batch * seq, d) with the Shape / Gather / Unsqueeze
/ Concat / Reshape pattern of Fig. 4, so the Gemm shapes after it are known
only to a mixed abstract/concrete interpretation.  Device of stage p, tensor
rank h: p * tp + h.
"""


def gpt2_layers(batch, seq, d=768, heads=12, n_layers=2, tp=2, pp=2, dtype="Float16"):
    """Program text for n_layers decoder layers over pp * tp devices.
    Concrete input: %flat = [-1] (the Reshape target's first entry)."""
    if heads % tp or d % heads or n_layers % pp:
        raise ValueError("heads must split over tp, d over heads, layers over pp")
    hl, dh, ff = heads // tp, d // heads, 4 * d // tp
    B, S = batch, seq
    params = ["%%x: Tensor[%s, (%d, %d, %d), 0]" % (dtype, B, S, d), "%flat: Tensor[Int32, (1,), 0]"]
    lines = []
    per = n_layers // pp
    for h in range(tp):
        dev = h
        lines += ["%%shape_%d = Shape(%%x)" % h,
                  "%%two_%d = Constant[value = 2]()" % h,
                  "%%dm_%d = Gather[axis = 0](%%shape_%d, %%two_%d)" % (h, h, h),
                  "%%dmu_%d = Unsqueeze[axes = [0]](%%dm_%d)" % (h, h),
                  "%%tgt_%d = Concat[axis = 0](%%flat, %%dmu_%d)" % (h, h)]
        if dev == 0:
            lines.append("%%h_0_0 = Reshape(%%x, %%tgt_%d)" % h)
        else:
            lines.append("%%x_r%d = Send[device = %d](%%x)" % (h, dev))
            lines.append("%%h_0_%d = Reshape(%%x_r%d, %%tgt_%d)" % (h, h, h))
    for L in range(n_layers):
        p = L // per
        for h in range(tp):
            dev = p * tp + h
            for w, shp in (("ln1", "(%d,)" % d), ("qkv", "(%d, %d)" % (d, 3 * hl * dh)),
                           ("proj", "(%d, %d)" % (hl * dh, d)), ("ln2", "(%d,)" % d),
                           ("fc1", "(%d, %d)" % (d, ff)), ("fc2", "(%d, %d)" % (ff, d))):
                params.append("%%W%s_%d_%d: Tensor[%s, %s, %d] keep" % (w, L, h, dtype, shp, dev))
            x = "%%h_%d_%d" % (L, h)
            q = "%d_%d" % (L, h)
            lines += [
                # concrete reshape targets of the attention block
                "%%c5_%s = Constant[value = [%d, %d, 3, %d, %d]]()" % (q, B, S, hl, dh),
                "%%c2_%s = Constant[value = [%d, %d]]()" % (q, B * S, hl * dh),
                "%%a_%s = LayerNormalization(%s, %%Wln1_%s, %%Wln1_%s)" % (q, x, q, q),
                "%%qkv_%s = Gemm(%%a_%s, %%Wqkv_%s)" % (q, q, q),
                "%%qkv5_%s = Reshape(%%qkv_%s, %%c5_%s)" % (q, q, q),
                "%%qkvt_%s = Transpose[perm = [2, 0, 3, 1, 4]](%%qkv5_%s)" % (q, q),
                "%%q_%s, %%k_%s, %%v_%s = Split[axis = 0, split = [1, 1, 1]](%%qkvt_%s)" % (q, q, q, q),
                "%%kt_%s = Transpose[perm = [0, 1, 2, 4, 3]](%%k_%s)" % (q, q),
                "%%sc_%s = MatMul(%%q_%s, %%kt_%s)" % (q, q, q),
                "%%pr_%s = Softmax[axis = -1](%%sc_%s)" % (q, q),
                "%%o_%s = MatMul(%%pr_%s, %%v_%s)" % (q, q, q),
                "%%ot_%s = Transpose[perm = [0, 1, 3, 2, 4]](%%o_%s)" % (q, q),
                "%%of_%s = Reshape(%%ot_%s, %%c2_%s)" % (q, q, q),
                "%%y_%s = Gemm(%%of_%s, %%Wproj_%s)" % (q, q, q),
            ]
        ys = ", ".join("%%y_%d_%d" % (L, h) for h in range(tp))
        outs = ", ".join("%%yr_%d_%d" % (L, h) for h in range(tp))
        lines.append("%s = AllReduce(%s)" % (outs, ys) if tp > 1 else "%%yr_%d_0 = Identity(%%y_%d_0)" % (L, L))
        for h in range(tp):
            q = "%d_%d" % (L, h)
            lines += [
                "%%r_%s = Add(%%h_%s, %%yr_%s)" % (q, q, q),
                "%%b_%s = LayerNormalization(%%r_%s, %%Wln2_%s, %%Wln2_%s)" % (q, q, q, q),
                "%%f_%s = Gemm(%%b_%s, %%Wfc1_%s)" % (q, q, q),
                "%%g_%s = Gelu(%%f_%s)" % (q, q),
                "%%m_%s = Gemm(%%g_%s, %%Wfc2_%s)" % (q, q, q),
            ]
        ms = ", ".join("%%m_%d_%d" % (L, h) for h in range(tp))
        outs = ", ".join("%%mr_%d_%d" % (L, h) for h in range(tp))
        lines.append("%s = AllReduce(%s)" % (outs, ms) if tp > 1 else "%%mr_%d_0 = Identity(%%m_%d_0)" % (L, L))
        for h in range(tp):
            q = "%d_%d" % (L, h)
            nxt = "%%h_%d_%d" % (L + 1, h)
            if L + 1 < n_layers and (L + 1) // per != p:
                lines.append("%%z_%s = Add(%%r_%s, %%mr_%s)" % (q, q, q))
                lines.append("%s = Send[device = %d](%%z_%s)" % (nxt, ((L + 1) // per) * tp + h, q))
            else:
                lines.append("%s = Add(%%r_%s, %%mr_%s)" % (nxt, q, q))
    rets = ", ".join("%%h_%d_%d" % (n_layers, h) for h in range(tp))
    return "func gpt2(%s)\n%s\nreturn %s\n" % (", ".join(params), "\n".join(lines), rets)
