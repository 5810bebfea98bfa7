"""fp64 CPU oracle for one host's share of APB prefill attention.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import it.  The product path (the
HIP library and its Python binding) never calls it and shares no code with it.
"""
from .apb_oracle import (  # noqa: F401
    bf16_to_f64,
    visible_end,
    assemble_kv,
    attention_ref,
    topk_ref,
    gather_ref,
    compress_ref,
    simulate_hosts_ref,
    attention_flops,
)
from .decode_oracle import (  # noqa: F401
    decode_attention_ref,
    merge_ref,
    stage2_ref,
)
from .scorer_oracle import (  # noqa: F401
    scorer_features,
    silu,
    retaining_scores_ref,
    scorer_flops,
)
from .layer_oracle import (  # noqa: F401
    rmsnorm_ref,
    rope_ref,
    swiglu_ffn_ref,
    qkv_ref,
    layer_ref,
    layer_flops,
    apb_table_flops_per_layer,
)
