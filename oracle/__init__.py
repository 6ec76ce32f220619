"""fp64 CPU oracle for ragged paged-KV decode / append attention.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run anything here.  The library
(``paper_2606_03077_amd``) never imports it and shares no code with it: the oracle reads
the *logical* paged format produced by the input generator, never the library's device
layout, and re-derives everything it computes from the definitions below.

What it computes
----------------
The paper (Sec. 1, Sec. 2.1 and App. A.1) treats rollout as autoregressive decoding
that is bound by memory bandwidth and KV-cache pressure, with tool outputs appended to
the context mid-trajectory (Sec. 5, Phase 2 and Step 3), but it never writes attention
down; its engine (vLLM, Sec. 6) does scaled dot-product softmax attention over a paged
KV cache.  The oracle is therefore the plain definition, evaluated directly in float64:

    z_j = s * <q, k_j>,  o = sum_j softmax(z)_j v_j,  LSE = log(sum_j exp(z_j))

with grouped query heads (query head h reads KV head h // G), page indirection through
a block table, and, for appended chunks, causal visibility of keys up to and including
the query's own position.  The split plan (``oracle.plan``) re-implements the library's
published partitioning rule in plain Python integers.

Every function names the passage or reading it follows; the readings the paper leaves
open are listed in the design notes of the repository.
"""
from .attention import (  # noqa: F401
    bf16_bits_to_f64,
    gather_tokens,
    attend,
    decode_ref,
    append_ref,
    write_new_tokens,
    merge_ref,
)
from .plan import plan_ref, PlanParams, UNIT_FIELDS  # noqa: F401
from .migration import reshard_heads, request_pages, query_heads_of_shard  # noqa: F401
from .cost_model import (  # noqa: F401
    ce_fit_ref, mape_ref, poly_sum_ref, instance_cost, rollout_dp_ref, partition_makespan,
)
from .scheduler import PrefixTreeRef, route_ref  # noqa: F401
