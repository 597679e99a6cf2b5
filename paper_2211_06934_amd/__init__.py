"""MI355X-native differentiable-Adam hot path (TorchOpt, arXiv 2211.06934).

The product is the HIP library ``libdiffopt.so`` behind ``include/diffopt.h``:
fused Adam forward, its fused VJP, a K-step unrolled driver, tree
flatten/unflatten through a segment table, the leaf-direct ("tree map") form
of the step that works on the leaves without flattening, fused differentiable
SGD-momentum and RMSProp (flat and leaf-direct), and the zero-order (ES)
estimator.  ``diffopt`` is its thin Python binding (same entry points),
``tree`` the host-side container walk and ``autograd`` the
torch.autograd.Functions and meta-optimizers over the fused steps.  Importing
the package loads the library and raises ImportError if it has not been
built.
"""
from . import diffopt
from .diffopt import (DiffoptError, SegTable, adam_bwd, adam_bwd_tree, adam_fwd, adam_fwd_tree,
                      adam_unrolled_bwd, adam_unrolled_bwd_tree, adam_unrolled_fwd,
                      adam_unrolled_fwd_tree, last_error, segtable_create, segtable_destroy,
                      segtable_nseg, segtable_total, tree_flatten, tree_unflatten,
                      tree_flatten_batch, tree_unflatten_batch,
                      sgd_fwd, sgd_bwd, rmsprop_fwd, rmsprop_bwd, es_perturb, es_estimate,
                      es_perturb_gaussian, es_estimate_gaussian, es_weights,
                      sgd_fwd_tree, sgd_bwd_tree, rmsprop_fwd_tree, rmsprop_bwd_tree)
from . import tree
from . import autograd
from .autograd import (AdamFn, AdamHyper, AdamState, AdamTreeFn, FlatAdam, MetaAdam, MetaRMSProp, MetaSGD,
                       RMSPropHyper, RMSPropTreeFn, SGDHyper, SGDTreeFn, ZeroOrderFn, es_gradient)

__all__ = [
    "diffopt", "tree", "autograd", "DiffoptError", "SegTable", "adam_bwd", "adam_fwd",
    "adam_unrolled_bwd", "adam_unrolled_fwd", "adam_fwd_tree", "adam_bwd_tree",
    "adam_unrolled_fwd_tree", "adam_unrolled_bwd_tree", "sgd_fwd", "sgd_bwd", "rmsprop_fwd", "rmsprop_bwd",
    "sgd_fwd_tree", "sgd_bwd_tree", "rmsprop_fwd_tree", "rmsprop_bwd_tree",
    "es_perturb", "es_estimate", "es_perturb_gaussian", "es_estimate_gaussian", "es_weights", "last_error", "segtable_create", "segtable_destroy",
    "segtable_nseg", "segtable_total", "tree_flatten", "tree_unflatten", "tree_flatten_batch",
    "tree_unflatten_batch", "AdamFn", "AdamHyper",
    "AdamState", "FlatAdam", "AdamTreeFn", "MetaAdam", "SGDHyper", "SGDTreeFn", "MetaSGD", "RMSPropHyper",
    "RMSPropTreeFn", "MetaRMSProp", "ZeroOrderFn", "es_gradient",
]
