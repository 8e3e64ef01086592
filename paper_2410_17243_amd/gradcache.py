"""Gradient-cache driver around the tiled loss (the training setup of Sec. 4.1,
which pairs the loss with Gradient Cache so that encoder memory does not grow
with the batch).

One step, for encoders f_I, f_T and inputs x_I, x_T of b samples:
  1. embed every chunk of `chunk` samples with no autograd graph, into
     contiguous [b, d] buffers of the loss's input type;
  2. the loss and its gradients with respect to the embeddings and the scale,
     by the HIP kernels (infcl_fwd / infcl_bwd): memory linear in b;
  3. embed every chunk again, this time with a graph, and backpropagate the
     cached embedding gradient of that chunk into the encoder parameters,
     which accumulate over the chunks.
Peak memory is one chunk's activations, the embeddings and their gradients,
and the loss's workspace, instead of the activations of all b samples.

The encoders here are whatever torch modules the caller passes; the tests use
small random-initialised ones (there are no trained weights or datasets here).
Only the loss runs in the library's kernels; the encoders are ordinary torch.
"""

from __future__ import annotations

from . import clip_loss_bwd, clip_loss_fwd, workspace_for


def chunks(b: int, chunk: int):
    """[r0, r1) ranges of at most `chunk` samples covering [0, b)."""
    if chunk < 1:
        raise ValueError(f"chunk must be >= 1, got {chunk}")
    return [(r0, min(b, r0 + chunk)) for r0 in range(0, b, chunk)]


def gradcache_step(enc_img, enc_txt, x_img, x_txt, scale, chunk: int, emb_dtype=None):
    """Accumulate d loss / d parameters of both encoders (into .grad) and return
    (loss, dscale) for one step of b = x_img.shape[0] samples.

    enc_img / enc_txt map [n, *] inputs to [n, d] embeddings (any float type;
    they are cast to emb_dtype, default bfloat16, before the loss).  scale is
    a float32 device tensor of one element; its gradient is returned, not
    accumulated (the caller owns how the scale is parametrised)."""
    import torch

    emb_dtype = emb_dtype or torch.bfloat16
    b = x_img.shape[0]
    if x_txt.shape[0] != b:
        raise ValueError("x_img and x_txt must hold the same number of samples")
    ranges = chunks(b, chunk)
    # 1. embeddings, chunk by chunk, without graphs
    with torch.no_grad():
        first = enc_img(x_img[ranges[0][0]:ranges[0][1]])
        d = first.shape[1]
        E_I = torch.empty((b, d), dtype=emb_dtype, device=first.device)
        E_T = torch.empty((b, d), dtype=emb_dtype, device=first.device)
        E_I[ranges[0][0]:ranges[0][1]] = first.to(emb_dtype)
        for k, (r0, r1) in enumerate(ranges):
            if k:
                E_I[r0:r1] = enc_img(x_img[r0:r1]).to(emb_dtype)
            E_T[r0:r1] = enc_txt(x_txt[r0:r1]).to(emb_dtype)
        del first
    # 2. the loss and the embedding gradients (HIP kernels)
    sc = scale.reshape(()).to(torch.float32).contiguous()
    ws = workspace_for(E_I)
    f = clip_loss_fwd(E_I, E_T, sc, workspace=ws)
    dI, dT, dscale = clip_loss_bwd(E_I, E_T, sc, f, workspace=ws)
    # 3. re-embed with graphs and backpropagate the cached gradients
    for r0, r1 in ranges:
        out = enc_img(x_img[r0:r1])
        out.to(emb_dtype).to(torch.float32).backward(dI[r0:r1])
        out = enc_txt(x_txt[r0:r1])
        out.to(emb_dtype).to(torch.float32).backward(dT[r0:r1])
    return f["loss"], dscale
