"""Layer tables of the network-shaped stacks (shapes only, no weights).

Activations are numbered: 0 is the stack input, layer i writes activation
i + 1.  A layer reads activation `src` and, if `res` is set, adds activation
`res` before its activation function (the fused epilogue computes
act(conv + bias + residual)).

* ResNet-50 v1.5 at 224 x 224: 7x7/2 stem, 3x3/2 max pool, bottlenecks
  1x1 -> 3x3 (stride here) -> 1x1 with widths 64..512 (outputs 256..2048),
  projection shortcuts on the first block of each stage, ReLU after c1, c2
  and after (c3 + shortcut).  53 convolutions, no classifier head.
* MobileNetV2 at 224 x 224: 3x3/2 stem, inverted residual blocks
  (expansion t, output c, repeats n, stride s) with ReLU6 after the expand
  and depthwise convs, a linear projection, a residual when stride 1 and
  c_in == c_out, and the final 1x1 320 -> 1280.  52 convolutions (17
  depthwise), no head.
* Transformer FFN blocks: x <- x + W2 ReLU(W1 x) with hidden 768 -> 3072 ->
  768 over seq x batch tokens, 12 blocks, no normalisation.
Biases are zero everywhere (has_bias = 0).
"""
from dataclasses import dataclass, field

ACT_NONE, ACT_RELU, ACT_RELU6 = 0, 1, 2


@dataclass
class Layer:
    name: str
    kind: str                 # "conv", "fc" or "maxpool"
    src: int
    shape: dict = field(default_factory=dict)
    act: int = ACT_NONE
    res: int = None

    @property
    def depthwise(self):
        s = self.shape
        return self.kind == "conv" and s["groups"] > 1 and s["groups"] == s["cin"] == s["cout"]


def _out(h, k, s, p):
    return (h + 2 * p - k) // s + 1


def conv(name, src, n, cin, h, w, cout, k, s, p, act, groups=1, res=None):
    return Layer(name, "conv", src, dict(n=n, cin=cin, h=h, w=w, cout=cout, kh=k, kw=k, sh=s,
                                         sw=s, ph=p, pw=p, groups=groups), act, res)


def resnet50(n):
    L = []
    L.append(conv("stem", 0, n, 3, 224, 224, 64, 7, 2, 3, ACT_RELU))
    L.append(Layer("maxpool", "maxpool", 1, dict(n=n, c=64, h=112, w=112, k=3, s=2, p=1)))
    cur, cin, hw = 2, 64, 56
    for si, (width, blocks, stride) in enumerate(((64, 3, 1), (128, 4, 2), (256, 6, 2),
                                                  (512, 3, 2))):
        for b in range(blocks):
            s = stride if b == 0 else 1
            ho = _out(hw, 3, s, 1)
            tag = f"s{si + 1}b{b + 1}"
            L.append(conv(f"{tag}.c1", cur, n, cin, hw, hw, width, 1, 1, 0, ACT_RELU))
            c1 = len(L)
            L.append(conv(f"{tag}.c2", c1, n, width, hw, hw, width, 3, s, 1, ACT_RELU))
            c2 = len(L)
            if b == 0:
                L.append(conv(f"{tag}.proj", cur, n, cin, hw, hw, 4 * width, 1, s, 0, ACT_NONE))
                short = len(L)
            else:
                short = cur
            L.append(conv(f"{tag}.c3", c2, n, width, ho, ho, 4 * width, 1, 1, 0, ACT_RELU,
                          res=short))
            cur, cin, hw = len(L), 4 * width, ho
    return L


MBV2_BLOCKS = ((1, 16, 1, 1), (6, 24, 2, 2), (6, 32, 3, 2), (6, 64, 4, 2), (6, 96, 3, 1),
               (6, 160, 3, 2), (6, 320, 1, 1))


def mobilenet_v2(n):
    L = [conv("stem", 0, n, 3, 224, 224, 32, 3, 2, 1, ACT_RELU6)]
    cur, cin, hw = 1, 32, 112
    for bi, (t, c, reps, stride) in enumerate(MBV2_BLOCKS):
        for r in range(reps):
            s = stride if r == 0 else 1
            hidden = cin * t
            tag = f"b{bi + 1}.{r + 1}"
            src = cur
            if t != 1:
                L.append(conv(f"{tag}.expand", src, n, cin, hw, hw, hidden, 1, 1, 0, ACT_RELU6))
                src = len(L)
            ho = _out(hw, 3, s, 1)
            L.append(conv(f"{tag}.dw", src, n, hidden, hw, hw, hidden, 3, s, 1, ACT_RELU6,
                          groups=hidden))
            L.append(conv(f"{tag}.project", len(L), n, hidden, ho, ho, c, 1, 1, 0, ACT_NONE,
                          res=cur if (s == 1 and cin == c) else None))
            cur, cin, hw = len(L), c, ho
    L.append(conv("last", cur, n, cin, hw, hw, 1280, 1, 1, 0, ACT_RELU6))
    return L


def ffn(tokens=2048, hidden=768, inner=3072, blocks=12):
    L = []
    cur = 0
    for b in range(blocks):
        L.append(Layer(f"ffn{b + 1}.fc1", "fc", cur, dict(m=tokens, k=hidden, n=inner), ACT_RELU))
        L.append(Layer(f"ffn{b + 1}.fc2", "fc", len(L), dict(m=tokens, k=inner, n=hidden),
                       ACT_NONE, res=cur))
        cur = len(L)
    return L


def input_shape(layers):
    """NHWC (or [m, k]) shape of activation 0."""
    s = layers[0].shape
    if layers[0].kind == "fc":
        return (s["m"], s["k"])
    return (s["n"], s["h"], s["w"], s["cin"])


def output_shape(layer):
    s = layer.shape
    if layer.kind == "fc":
        return (s["m"], s["n"])
    if layer.kind == "maxpool":
        return (s["n"], _out(s["h"], s["k"], s["s"], s["p"]), _out(s["w"], s["k"], s["s"], s["p"]),
                s["c"])
    return (s["n"], _out(s["h"], s["kh"], s["sh"], s["ph"]), _out(s["w"], s["kw"], s["sw"], s["pw"]),
            s["cout"])
