"""The sharded loss of n GPUs, run as n shards on one device.

Each shard is one GPU's share of the batch (samples [r0, r0 + bs)): the C ABI's
infcl_fwd_shard / infcl_fwd_shard_finish / infcl_bwd_shard compute it with the
same kernels as the whole-batch entry points, on a rectangle of bs own rows by
b columns.  Here the n shards run one after another on one device, each with
its own workspace, and the three exchanges of a multi-GPU run become plain
device copies in the order a collective would deliver them:

  all-to-all   shard g receives, from every shard k, the column pairs of its
               own columns [r0_g, r0_g + bs_g) out of shard k's colpair;
  all-reduce   loss and dscale are the sums of the shards' shares;
  all-gather   lse_r, lse_c and aux of every shard, in sample order, feed the
               backward of every shard.

Every step of the loss runs in the HIP kernels; torch only provides buffers and
copies (argument marshalling).
"""

from __future__ import annotations

from . import (_dtype_code, infcl_bwd_shard, infcl_fwd_shard, infcl_fwd_shard_finish, workspace_for)


def shard_bounds(b: int, n: int, align: int = 32):
    """Split [0, b) into n contiguous shards whose starts are multiples of `align`
    (the last shard takes the remainder)."""
    if n < 1 or n > b:
        raise ValueError(f"need 1 <= n <= b, got n={n}, b={b}")
    step = -(-b // n)
    step = -(-step // align) * align
    bounds = []
    r0 = 0
    while r0 < b:
        bs = min(step, b - r0)
        bounds.append((r0, bs))
        r0 += bs
    return bounds


def sharded_forward_backward(img, txt, scale, n: int, dloss=None, on_step=None, workspaces=None, out=None):
    """Loss, per-sample outputs and gradients of the whole batch, computed as n
    shards.  Returns a dict with loss64 (sum of the shards' shares), lse_r, lse_c,
    aux ([3b], in infcl_fwd's layout), dimg, dtxt, dscale64 and the shard bounds.

    on_step(name), if given, is called after each shard call is enqueued (e.g.
    to synchronise and report progress on very large batches).  workspaces (one
    per shard) and out (a previous result) may be passed to reuse buffers."""
    import torch

    b, d = img.shape
    dev = img.device
    dt = _dtype_code(img)
    bounds = shard_bounds(b, n)
    ws = workspaces if workspaces is not None else [workspace_for(img) for _ in bounds]
    note = on_step or (lambda name: None)
    # 1. local sweeps: one pair per column over each shard's rows
    colpair = [torch.empty(2 * b, dtype=torch.float32, device=dev) for _ in bounds]
    for g, ((r0, bs), w, cp) in enumerate(zip(bounds, ws, colpair)):
        infcl_fwd_shard(img, txt, scale, r0, bs, cp, w)
        note(f"forward shard {g + 1}/{len(bounds)}")
    # 2. all-to-all of column pairs, 3. finish on the column owners
    if out is not None:
        lse_r, lse_c, aux, dimg, dtxt = out["lse_r"], out["lse_c"], out["aux"], out["dimg"], out["dtxt"]
    else:
        lse_r = torch.empty(b, dtype=torch.float32, device=dev)
        lse_c = torch.empty(b, dtype=torch.float32, device=dev)
        aux = torch.empty(3 * b, dtype=torch.float32, device=dev)
        dimg = torch.empty((b, d), dtype=torch.float32, device=dev)
        dtxt = torch.empty((b, d), dtype=torch.float32, device=dev)
    loss_parts = torch.empty(len(bounds), dtype=torch.float64, device=dev)
    for g, ((r0, bs), w) in enumerate(zip(bounds, ws)):
        recv = torch.empty((len(bounds), 2 * bs), dtype=torch.float32, device=dev)
        for k, cp in enumerate(colpair):
            recv[k, :bs] = cp[r0:r0 + bs]
            recv[k, bs:] = cp[b + r0:b + r0 + bs]
        o_lr = torch.empty(bs, dtype=torch.float32, device=dev)
        o_lc = torch.empty(bs, dtype=torch.float32, device=dev)
        o_aux = torch.empty(3 * bs, dtype=torch.float32, device=dev)
        infcl_fwd_shard_finish(b, d, dt, r0, bs, recv, scale, o_lr, o_lc, o_aux, loss_parts[g:g + 1], w)
        # 4. all-gather of the per-sample outputs
        lse_r[r0:r0 + bs] = o_lr
        lse_c[r0:r0 + bs] = o_lc
        for k in range(3):
            aux[k * b + r0:k * b + r0 + bs] = o_aux[k * bs:(k + 1) * bs]
    note("forward finished")
    # 5. backward shards
    ds_parts = torch.empty(len(bounds), dtype=torch.float64, device=dev)
    if dloss is not None:
        dloss = dloss.reshape(()).to(torch.float32).contiguous()
    for g, ((r0, bs), w) in enumerate(zip(bounds, ws)):
        infcl_bwd_shard(img, txt, scale, r0, bs, lse_r, lse_c, aux, dloss, dimg[r0:r0 + bs], dtxt[r0:r0 + bs],
                        ds_parts[g:g + 1], w)
        note(f"backward shard {g + 1}/{len(bounds)}")
    return {
        "loss64": loss_parts.sum(), "loss_parts": loss_parts, "lse_r": lse_r, "lse_c": lse_c, "aux": aux,
        "dimg": dimg, "dtxt": dtxt, "dscale64": ds_parts.sum(), "dscale_parts": ds_parts, "bounds": bounds,
    }
