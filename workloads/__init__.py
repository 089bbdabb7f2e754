"""Seeded synthetic inputs for the token-tree verification pass.

This package is the only code shared by the CPU oracle side (tests, the
oracle's CPU timing) and the GPU side (binding, bench).  It holds model
shapes, random-weight generation, prefix and draft-token draws and tree
shapes.  It contains none of the method's arithmetic: no norm, attention,
projection, argmax or accept logic.

The paper's own workloads need trained models and datasets (T5/mT5/Bart/GPT2,
Vicuna/LLaMa2, translation/QA/summarisation corpora, §4.1 and Table 3).
Random-weight LLaMA-shaped decoders and uniform token draws stand in for them.
"""

from .configs import ModelShape, Workload, MODELS, WORKLOADS, get_workload  # noqa: F401
from .rng import hash_uniform16, tensor_key  # noqa: F401
from .weights import ModelWeights, make_weights  # noqa: F401
from .trees import (  # noqa: F401
    chain_tree,
    complete_tree,
    random_tree,
    tree_depths,
    draw_tokens,
    make_tree,
    plant_path,
    draft_tree,
)
