"""A whole quantized network on the GPU: the CIFAR-10-shaped QNN of the
paper's end-to-end evaluation (Sec. V-E): three 5x5 convolutions with
requantization + ReLU clip, each followed by 2x2 max-pooling, then a fully
connected classifier with int32 logits.  Every layer is one library call on
one stream; activations stay in device memory between calls.
"""
from . import qnn


def cifar_forward(x, n, bits, cin, convs, fc, clip, stream=None, keep=False):
    """Run the network on packed NHWC input `x` (n x 32 x 32 x cin codes).

    convs: list of dicts with device tensors "w", "bias", "mult", "shift" and
    ints "m", "k", "pad"; fc: dict with "w", "bias", "m".  Returns the int32
    logits [n, 1, 1, m] (and the list of intermediate activations if keep).
    """
    h = w = 32
    c = cin
    acts = []
    for cv in convs:
        y = qnn.conv2d(x, (n, h, w, c), bits, cv["w"], cv["m"], cv["k"], cv["k"], (1, 1),
                       (cv["pad"], cv["pad"]), "requant", bias=cv["bias"], mult=cv["mult"],
                       shift=cv["shift"], clip=clip, stream=stream)
        h = (h + 2 * cv["pad"] - cv["k"]) + 1
        w = (w + 2 * cv["pad"] - cv["k"]) + 1
        c = cv["m"]
        x = qnn.maxpool2d(y, (n, h, w, c), bits, 2, 2, 2, 2, stream=stream)
        h //= 2
        w //= 2
        if keep:
            acts += [y, x]
    logits = qnn.linear(x, (n, h, w, c), bits, fc["w"], fc["m"], "raw32", bias=fc["bias"],
                        stream=stream)
    return (logits, acts) if keep else logits
