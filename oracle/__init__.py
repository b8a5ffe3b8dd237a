"""fp64 CPU oracle of the EE-Tuning exit-head step -- TEST INFRASTRUCTURE ONLY.

Only tests, the smoke check and the benchmark's CPU-baseline leg import this
package.  The product path never does.
"""

from .ee_oracle import (  # noqa: F401
    EXIT_EMBEDDING, EXIT_MLP, EXIT_NORM, Exit, ExitResult, confidence,
    exit_backward, exit_forward, exit_step, exit_step_sampled, layer_stats,
    layernorm_backward, log_sum_exp, logit_grad, multi_exit_step, norm_forward,
    rms_inv, rmsnorm_backward, row_weights, sigmoid, silu, silu_grad, softmax, token_nll,
    CHUNK_ROWS,
)


def exits_from_batch(batch):
    """Decode a workloads.Batch's stored parameters into float64 oracle exits."""
    from workloads import decode

    out = []
    for p in batch.exits:
        dec = (lambda a: None if a is None else decode(a))
        out.append(Exit(kind=p.kind, w_out=dec(p.w_out), gamma=dec(p.gamma),
                        gamma_mlp=dec(p.gamma_mlp), w_gate=dec(p.w_gate),
                        w_up=dec(p.w_up), w_down=dec(p.w_down),
                        eps=batch.workload.eps, norm=batch.workload.norm,
                        beta=dec(getattr(p, "beta", None))))
    return out
