"""MI355X-native batched verification step of confidence-scheduled speculative decoding.

Three stages, each a hand-written HIP kernel for gfx950 behind the C ABI in
``include/dspark.h``: the hardware-aware prefix scheduler, ragged paged verify
attention and speculative acceptance; upstream of them, the drafter's
sequential stage (Markov and RNN heads), and input checks of the device-side
values.  The binding (``paper_2607_05147_amd.dspark``)
is loaded on first use so that the input generator (``synth``) can be imported
without the GPU library.
"""

_BINDING_NAMES = (
    "dspark_abi_version", "dspark_last_error", "dspark_schedule", "dspark_verify_attn",
    "dspark_accept", "dspark_schedule_workspace_size", "dspark_verify_attn_workspace_size",
    "dspark_accept_workspace_size", "dspark_schedule_noalloc", "dspark_schedule_capacity",
    "dspark_schedule_topk", "dspark_markov_draft", "dspark_markov_draft_workspace_size",
    "dspark_rnn_draft", "dspark_rnn_draft_workspace_size", "check_verify_inputs",
    "check_accept_inputs", "check_schedule_inputs", "check_draft_inputs", "debug_checks", "DSparkError",
)


def __getattr__(name):
    if name in _BINDING_NAMES:
        from . import dspark
        return getattr(dspark, name)
    raise AttributeError(name)
