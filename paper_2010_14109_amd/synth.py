"""Seeded synthetic workloads: network descriptions and input/parameter bytes.

This module is shared by the product path and by the CPU oracle, so it holds
no part of the out-of-core method: no function sequence, no byte accounting,
no scheduling, no layer arithmetic.  It only states *which* network is trained
(layer kinds and their hyper-parameters, in topological order) and draws the
random bytes fed to both sides:

* data    -- ``numpy.random.Generator(PCG64(0))``: ``x`` as standard normal
             float32, then the labels as ``integers(0, classes)`` (int32);
* weights -- ``numpy.random.Generator(PCG64(1))``: He-normal fan-in for conv
             and dense weights, zero biases, BatchNorm gamma = 1, beta = 0.

Layouts are those of the library boundary: images are NHWC, conv weights are
``[K, R, S, C]`` (output channel, filter row, filter column, input channel),
dense weights are ``[out, in]``; token batches are ``[B, T]`` int32 and the
transformer's activations are ``[B T, features]``.  Transformer weights are
drawn N(0, 0.02).

The workloads stand in for the ones the paper trains (ResNet-50 on 224x224
ImageNet batches, Section 5.1 and Table 1) plus smaller networks of the same
layer kinds; ImageNet itself is not used.
"""

from __future__ import annotations

import numpy as np

# --------------------------------------------------------------------------
# network descriptions (plain data)
# --------------------------------------------------------------------------


def mlp(batch=256, width=1024, depth=8, classes=10, lr=0.01, momentum=0.0):
    """``depth`` dense layers of ``width`` with ReLU between them, last one to ``classes``."""
    layers = []
    prev = "x"
    for i in range(depth):
        out = classes if i == depth - 1 else width
        layers.append({"name": f"fc{i + 1}", "op": "linear", "in": [prev],
                       "in_features": width, "out_features": out})
        prev = f"fc{i + 1}"
        if i != depth - 1:
            layers.append({"name": f"relu{i + 1}", "op": "relu", "in": [prev]})
            prev = f"relu{i + 1}"
    return {"name": f"mlp{depth}_w{width}_b{batch}", "input": [batch, width],
            "classes": classes, "layers": layers, "logits": prev,
            "optimizer": {"lr": lr, "momentum": momentum}}


def plain_cnn(batch=128, channels=64, depth=10, hw=32, in_ch=3, classes=10,
              lr=0.01, momentum=0.0):
    """``depth`` x [conv3x3 s1 p1 + BatchNorm + ReLU], global average pool, dense head."""
    layers = []
    prev = "x"
    cin = in_ch
    for i in range(depth):
        layers.append({"name": f"conv{i + 1}", "op": "conv", "in": [prev], "cin": cin,
                       "cout": channels, "k": 3, "stride": 1, "pad": 1})
        layers.append({"name": f"bn{i + 1}", "op": "bn", "in": [f"conv{i + 1}"], "c": channels})
        layers.append({"name": f"relu{i + 1}", "op": "relu", "in": [f"bn{i + 1}"]})
        prev = f"relu{i + 1}"
        cin = channels
    layers.append({"name": "gap", "op": "avgpool", "in": [prev]})
    layers.append({"name": "fc", "op": "linear", "in": ["gap"], "in_features": channels,
                   "out_features": classes})
    return {"name": f"cnn{depth}_c{channels}_b{batch}", "input": [batch, hw, hw, in_ch],
            "classes": classes, "layers": layers, "logits": "fc",
            "optimizer": {"lr": lr, "momentum": momentum}}


def resnet(batch=256, hw=224, classes=1000, blocks=(3, 4, 6, 3), width=64,
           lr=0.01, momentum=0.9):
    """Bottleneck ResNet (ResNet-50 for blocks (3,4,6,3)); stride on the 3x3 conv."""
    layers = []

    def conv_bn(name, src, cin, cout, k, stride, pad, relu=True):
        layers.append({"name": f"{name}.conv", "op": "conv", "in": [src], "cin": cin,
                       "cout": cout, "k": k, "stride": stride, "pad": pad})
        layers.append({"name": f"{name}.bn", "op": "bn", "in": [f"{name}.conv"], "c": cout})
        if relu:
            layers.append({"name": f"{name}.relu", "op": "relu", "in": [f"{name}.bn"]})
            return f"{name}.relu"
        return f"{name}.bn"

    prev = conv_bn("stem", "x", 3, width, 7, 2, 3)
    layers.append({"name": "stem.pool", "op": "maxpool", "in": [prev], "k": 3, "stride": 2,
                   "pad": 1})
    prev = "stem.pool"
    cin = width
    for stage, nblocks in enumerate(blocks):
        mid = width * (2 ** stage)
        cout = mid * 4
        for b in range(nblocks):
            stride = 2 if (b == 0 and stage > 0) else 1
            base = f"s{stage + 1}b{b + 1}"
            h = conv_bn(f"{base}.a", prev, cin, mid, 1, 1, 0)
            h = conv_bn(f"{base}.b", h, mid, mid, 3, stride, 1)
            h = conv_bn(f"{base}.c", h, mid, cout, 1, 1, 0, relu=False)
            if b == 0:
                sc = conv_bn(f"{base}.down", prev, cin, cout, 1, stride, 0, relu=False)
            else:
                sc = prev
            layers.append({"name": f"{base}.add", "op": "add", "in": [h, sc]})
            layers.append({"name": f"{base}.out", "op": "relu", "in": [f"{base}.add"]})
            prev = f"{base}.out"
            cin = cout
    layers.append({"name": "gap", "op": "avgpool", "in": [prev]})
    layers.append({"name": "fc", "op": "linear", "in": ["gap"], "in_features": cin,
                   "out_features": classes})
    depth = 2 + 3 * sum(blocks)
    return {"name": f"resnet{depth}_b{batch}_{hw}", "input": [batch, hw, hw, 3],
            "classes": classes, "layers": layers, "logits": "fc",
            "optimizer": {"lr": lr, "momentum": momentum}}


def transformer(batch=64, seq=512, d=1024, heads=16, ffn=4096, layers=48, vocab=32000,
                lr=0.01, momentum=0.0):
    """Pre-LN causal transformer encoder with learned positions and an untied LM head,
    trained on next-token cross-entropy."""
    L = [{"name": "embed", "op": "embed", "in": ["x"], "vocab": vocab, "d": d}]
    prev = "embed"
    for i in range(layers):
        b = f"l{i + 1}"
        L += [
            {"name": f"{b}.ln1", "op": "layernorm", "in": [prev]},
            {"name": f"{b}.qkv", "op": "linear", "in": [f"{b}.ln1"], "in_features": d,
             "out_features": 3 * d},
            {"name": f"{b}.attn", "op": "attention", "in": [f"{b}.qkv"], "heads": heads,
             "causal": True},
            {"name": f"{b}.proj", "op": "linear", "in": [f"{b}.attn"], "in_features": d,
             "out_features": d},
            {"name": f"{b}.res1", "op": "add", "in": [f"{b}.proj", prev]},
            {"name": f"{b}.ln2", "op": "layernorm", "in": [f"{b}.res1"]},
            {"name": f"{b}.fc1", "op": "linear", "in": [f"{b}.ln2"], "in_features": d,
             "out_features": ffn},
            {"name": f"{b}.gelu", "op": "gelu", "in": [f"{b}.fc1"]},
            {"name": f"{b}.fc2", "op": "linear", "in": [f"{b}.gelu"], "in_features": ffn,
             "out_features": d},
            {"name": f"{b}.res2", "op": "add", "in": [f"{b}.fc2", f"{b}.res1"]},
        ]
        prev = f"{b}.res2"
    L += [{"name": "lnf", "op": "layernorm", "in": [prev]},
          {"name": "head", "op": "linear", "in": ["lnf"], "in_features": d, "out_features": vocab}]
    return {"name": f"transformer{layers}_d{d}_b{batch}_t{seq}", "input": [batch, seq],
            "tokens": True, "classes": vocab, "layers": L, "logits": "head", "init": "normal",
            "optimizer": {"lr": lr, "momentum": momentum}}


def densenet(batch=64, hw=64, growth=32, blocks=(6, 12, 24, 16), stem=64, classes=10,
             lr=0.01, momentum=0.9):
    """DenseNet-shaped network (no bottleneck): inside a block every layer reads the channel
    concatenation of the stem or transition output and of every earlier layer's output
    (BN, ReLU, conv3x3 to ``growth`` channels), so each feature map is read by all later layers
    of its block.  Between blocks: concatenation, BN, ReLU, conv1x1 to half the channels,
    2x2 max pool.  Head: concatenation, BN, ReLU, global average pool, dense."""
    layers = [{"name": "stem", "op": "conv", "in": ["x"], "cin": 3, "cout": stem, "k": 3,
               "stride": 1, "pad": 1}]
    feats, chans = ["stem"], [stem]

    def gather(name):
        if len(feats) == 1:
            return feats[0]
        layers.append({"name": name, "op": "concat", "in": list(feats)})
        return name

    for b, n in enumerate(blocks):
        for i in range(n):
            base = f"b{b + 1}l{i + 1}"
            src = gather(f"{base}.cat")
            layers += [
                {"name": f"{base}.bn", "op": "bn", "in": [src], "c": sum(chans)},
                {"name": f"{base}.relu", "op": "relu", "in": [f"{base}.bn"]},
                {"name": f"{base}.conv", "op": "conv", "in": [f"{base}.relu"], "cin": sum(chans),
                 "cout": growth, "k": 3, "stride": 1, "pad": 1},
            ]
            feats.append(f"{base}.conv")
            chans.append(growth)
        c = sum(chans)
        base = f"t{b + 1}" if b + 1 < len(blocks) else "head"
        src = gather(f"{base}.cat")
        layers += [{"name": f"{base}.bn", "op": "bn", "in": [src], "c": c},
                   {"name": f"{base}.relu", "op": "relu", "in": [f"{base}.bn"]}]
        if b + 1 < len(blocks):
            layers += [
                {"name": f"{base}.conv", "op": "conv", "in": [f"{base}.relu"], "cin": c,
                 "cout": c // 2, "k": 1, "stride": 1, "pad": 0},
                {"name": f"{base}.pool", "op": "maxpool", "in": [f"{base}.conv"], "k": 2,
                 "stride": 2, "pad": 0},
            ]
            feats, chans = [f"{base}.pool"], [c // 2]
        else:
            layers += [{"name": "gap", "op": "avgpool", "in": [f"{base}.relu"]},
                       {"name": "fc", "op": "linear", "in": ["gap"], "in_features": c,
                        "out_features": classes}]
    return {"name": f"densenet{sum(blocks)}_g{growth}_b{batch}_{hw}",
            "input": [batch, hw, hw, 3], "classes": classes, "layers": layers, "logits": "fc",
            "optimizer": {"lr": lr, "momentum": momentum}}


def unet(batch=8, hw=256, base=64, depth=4, classes=8, lr=0.01, momentum=0.9):
    """U-Net-shaped segmentation network: ``depth`` encoder levels of two (conv3x3, BN, ReLU)
    followed by a 2x2 max pool, a bottleneck, and decoder levels that upsample (nearest, 2x),
    convolve to the level's width, concatenate the encoder output of the same level (a skip
    across the whole network) and apply two (conv3x3, BN, ReLU); a conv1x1 gives per-pixel
    logits, trained on per-pixel labels."""
    layers = []

    def cbr(name, src, cin, cout):
        layers.extend([
            {"name": f"{name}.conv", "op": "conv", "in": [src], "cin": cin, "cout": cout, "k": 3,
             "stride": 1, "pad": 1},
            {"name": f"{name}.bn", "op": "bn", "in": [f"{name}.conv"], "c": cout},
            {"name": f"{name}.relu", "op": "relu", "in": [f"{name}.bn"]}])
        return f"{name}.relu"

    prev, cin, skips = "x", 3, []
    for i in range(depth):
        c = base * 2 ** i
        prev = cbr(f"e{i + 1}a", prev, cin, c)
        prev = cbr(f"e{i + 1}b", prev, c, c)
        skips.append((prev, c))
        layers.append({"name": f"e{i + 1}.pool", "op": "maxpool", "in": [prev], "k": 2,
                       "stride": 2, "pad": 0})
        prev, cin = f"e{i + 1}.pool", c
    c = base * 2 ** depth
    prev = cbr("mid.a", prev, cin, c)
    prev = cbr("mid.b", prev, c, c)
    cin = c
    for i in reversed(range(depth)):
        skip, c = skips[i]
        layers.append({"name": f"d{i + 1}.up", "op": "upsample", "in": [prev]})
        prev = cbr(f"d{i + 1}u", f"d{i + 1}.up", cin, c)
        layers.append({"name": f"d{i + 1}.cat", "op": "concat", "in": [prev, skip]})
        prev = cbr(f"d{i + 1}a", f"d{i + 1}.cat", 2 * c, c)
        prev = cbr(f"d{i + 1}b", prev, c, c)
        cin = c
    layers.append({"name": "out", "op": "conv", "in": [prev], "cin": cin, "cout": classes, "k": 1,
                   "stride": 1, "pad": 0})
    return {"name": f"unet{depth}_c{base}_b{batch}_{hw}", "input": [batch, hw, hw, 3],
            "classes": classes, "dense_labels": True, "layers": layers, "logits": "out",
            "optimizer": {"lr": lr, "momentum": momentum}}


#: The workloads: name -> (network description, budget as a fraction of the
#: in-core peak).  The first five are the benchmark configurations; densenet
#: and unet are long-skip networks whose feature maps are read many times.
WORKLOADS = {
    "mlp": (lambda: mlp(), 0.40),
    "cnn": (lambda: plain_cnn(), 0.50),
    "resnet50_b256": (lambda: resnet(batch=256), 0.25),
    "resnet50_b1440": (lambda: resnet(batch=1440), 1.0 / 7.5),
    "transformer": (lambda: transformer(), 0.20),
    "densenet": (lambda: densenet(), 0.25),
    "unet": (lambda: unet(), 0.25),
}


def workload(name, **overrides):
    """Network description of a named workload, with keyword overrides (e.g. ``batch=8``)."""
    builders = {"mlp": mlp, "cnn": plain_cnn, "resnet50_b256": resnet,
                "resnet50_b1440": resnet, "transformer": transformer, "densenet": densenet,
                "unet": unet}
    defaults = {"resnet50_b256": {"batch": 256}, "resnet50_b1440": {"batch": 1440}}
    kw = dict(defaults.get(name, {}))
    kw.update(overrides)
    return builders[name](**kw)


def budget_fraction(name):
    return WORKLOADS[name][1]


# --------------------------------------------------------------------------
# seeded bytes
# --------------------------------------------------------------------------


def param_shapes(spec):
    """Parameter tensors of a network description, in layer order: ``[(name, shape)]``.

    The shapes are read off the layer hyper-parameters only.
    """
    out = []
    for L in spec["layers"]:
        if L["op"] == "embed":
            out.append((L["name"] + ".E", (L["vocab"], L["d"])))
            out.append((L["name"] + ".pos", (spec["input"][1], L["d"])))
        elif L["op"] == "layernorm":
            out.append((L["name"] + ".gamma", (_width(spec, L),)))
            out.append((L["name"] + ".beta", (_width(spec, L),)))
        elif L["op"] == "linear":
            out.append((L["name"] + ".W", (L["out_features"], L["in_features"])))
            out.append((L["name"] + ".b", (L["out_features"],)))
        elif L["op"] == "conv":
            out.append((L["name"] + ".W", (L["cout"], L["k"], L["k"], L["cin"])))
        elif L["op"] == "bn":
            out.append((L["name"] + ".gamma", (L["c"],)))
            out.append((L["name"] + ".beta", (L["c"],)))
    return out


def _width(spec, layer):
    """Feature width of a transformer LayerNorm: the model width of the embedding."""
    return next(L["d"] for L in spec["layers"] if L["op"] == "embed")


def make_inputs(spec, seed=0):
    """``(x, labels)``.  Images: x float32 of the input shape, labels int32 [N] uniform over
    the classes ([N H W], one per pixel, for per-pixel logits).  Tokens: ids [B, T + 1] uniform over the vocabulary; x = ids[:, :T] (int32)
    and the labels are the next tokens ids[:, 1:] flattened to [B T]."""
    g = np.random.Generator(np.random.PCG64(seed))
    if spec.get("tokens"):
        B, T = spec["input"]
        ids = g.integers(0, spec["classes"], size=(B, T + 1)).astype(np.int32)
        return np.ascontiguousarray(ids[:, :T]), np.ascontiguousarray(ids[:, 1:]).reshape(-1)
    x = g.standard_normal(size=tuple(spec["input"]), dtype=np.float32)
    n = int(np.prod(spec["input"][:3])) if spec.get("dense_labels") else spec["input"][0]
    labels = g.integers(0, spec["classes"], size=n).astype(np.int32)
    return x, labels


def make_params(spec, seed=1):
    """Initial parameters ``{name: float32 array}`` (He-normal fan-in, zero bias, BN 1/0)."""
    g = np.random.Generator(np.random.PCG64(seed))
    params = {}
    normal = spec.get("init") == "normal"
    for name, shape in param_shapes(spec):
        kind = name.rsplit(".", 1)[1]
        if normal and kind in ("W", "E", "pos"):
            params[name] = (g.standard_normal(size=shape, dtype=np.float32)
                            * np.float32(0.02)).astype(np.float32)
        elif kind == "W":
            fan_in = int(np.prod(shape[1:]))
            std = np.float32(np.sqrt(2.0 / fan_in))
            params[name] = (g.standard_normal(size=shape, dtype=np.float32) * std).astype(np.float32)
        elif kind == "gamma":
            params[name] = np.ones(shape, np.float32)
        else:  # bias or beta
            params[name] = np.zeros(shape, np.float32)
    return params


def normal_pool(n, seed, threads=16):
    """``n`` standard-normal float32 values drawn by ``threads`` PCG64 streams spawned from
    ``SeedSequence(seed)``, stream i filling the i-th of ``threads`` equal blocks.  The same
    (n, seed, threads) gives the same array on any host.  Large full-size test inputs are
    windows of one such pool."""
    from concurrent.futures import ThreadPoolExecutor
    out = np.empty(n, np.float32)
    streams = np.random.SeedSequence(seed).spawn(threads)
    step = -(-n // threads)

    def fill(i):
        block = out[i * step:(i + 1) * step]
        if block.size:
            np.random.Generator(np.random.PCG64(streams[i])).standard_normal(
                size=block.size, dtype=np.float32, out=block)

    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(fill, range(threads)))
    return out
