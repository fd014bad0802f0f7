"""MI355X-native batched latent-rollout evaluator (compiler world model).

The hot path (rollout, scoring, top-k; the tree-ensemble ranker; the
rollout loss and its gradients; the chunked transformer state encoder) runs
in hand-written gfx950 HIP kernels behind the C ABI of include/wm.h; this
package is the thin Python binding over it.
"""
from .binding import (  # noqa: F401
    GRAD_KEYS, KERNELS, NORMS, PRECISIONS, SYMBOLS, WMError, Forest, Model, TextModel,
    device_status, encode_init, encode_text, evaluate, evaluate_noalloc, grad_shapes, load_library,
    loss_workspace,
    phi_struct, rollout, rollout_loss, score, score_trees, timing_enable, timing_read, topk,
)


def model_dims(w) -> dict:
    """Model dims dict from an object with the workload fields (d, e, ...)."""
    return {k: getattr(w, k) for k in ("d", "e", "n_kinds", "n_params", "H", "C", "hw_dim",
                                       "feat_dim", "enc_hidden")}
