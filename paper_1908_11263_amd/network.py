"""A whole quantized network on the GPU: the CIFAR-10-shaped QNN of the
paper's end-to-end evaluation (Sec. V-E): three 5x5 convolutions with
requantization + ReLU clip, each followed by 2x2 max-pooling, then a fully
connected classifier with int32 logits.  Every layer is one library call on
one stream; activations stay in device memory between calls.
"""
from . import qnn


def cifar_forward(x, n, bits, cin, convs, fc, clip, stream=None, keep=False, fused=True):
    """Run the network on packed NHWC input `x` (n x 32 x 32 x cin codes).

    convs: list of dicts with device tensors "w", "bias", "mult", "shift" and
    ints "m", "k", "pad"; fc: dict with "w", "bias", "m".  Each convolution
    runs fused with its 2x2 max-pooling (qnn_conv2d_maxpool), or, with
    fused=False, as a convolution followed by a separate pooling.  Returns
    the int32 logits [n, 1, 1, m] (and the list of intermediate activations
    if keep: pooled outputs, preceded by the convolution outputs when not
    fused).
    """
    h = w = 32
    c = cin
    acts = []
    for cv in convs:
        args = (bits, cv["w"], cv["m"], cv["k"], cv["k"], (1, 1), (cv["pad"], cv["pad"]), "requant")
        kw = dict(bias=cv["bias"], mult=cv["mult"], shift=cv["shift"], clip=clip, stream=stream)
        ho = (h + 2 * cv["pad"] - cv["k"]) + 1
        wo = (w + 2 * cv["pad"] - cv["k"]) + 1
        if fused:
            x = qnn.conv2d_maxpool(x, (n, h, w, c), *args, **kw)
            if keep:
                acts.append(x)
        else:
            y = qnn.conv2d(x, (n, h, w, c), *args, **kw)
            x = qnn.maxpool2d(y, (n, ho, wo, cv["m"]), bits, 2, 2, 2, 2, stream=stream)
            if keep:
                acts += [y, x]
        h, w, c = ho // 2, wo // 2, cv["m"]
    logits = qnn.linear(x, (n, h, w, c), bits, fc["w"], fc["m"], "raw32", bias=fc["bias"],
                        stream=stream)
    return (logits, acts) if keep else logits
