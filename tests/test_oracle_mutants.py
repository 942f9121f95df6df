"""Plant mistakes in a copy of the oracle and require the pins to catch each.

Every mutant is a textual edit of ``oracle/cpdp_oracle.c`` compiled into a
temporary library (CPU only).  A mutant that passes every pin would mean the
pins cannot tell that mistake from the method, so the test fails.  Only pins
that check the oracle against something other than itself count:
pin_general_sgd_matches_plain compares two oracle functions with each other,
so a mistake made in both would pass it, and it is left out here.
"""
import os

import pytest

import oracle
import oracle_pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "cpdp_oracle.c")

# (name, old text, new text, which occurrence of old text to replace)
MUTANTS = [
    ("local_drops_mu", "mu * mom[k] + grads[k]", "mom[k] + grads[k]", 0),
    ("local_steps_on_grad",
     "params[k] = store_as(param_dt, params[k] - lr * buf);",
     "params[k] = store_as(param_dt, params[k] - lr * grads[k]);", 0),
    ("gbar_not_divided", "gsum / (double)W", "gsum", 0),
    ("sync_uses_local_grad", "mu * mom[k] + gbar", "mu * mom[k] + grads[k]", 0),
    ("sync_drops_mu", "mu * mom[k] + gbar", "mom[k] + gbar", 0),
    ("sync_buffer_not_stored", "mom[k] = buf;\n            double x",
     "double x", 0),
    ("u_sign_flipped", "(ref - avg) / lr", "(avg - ref) / lr", 0),
    ("u_drops_lr", "(ref - avg) / lr", "(ref - avg)", 0),
    ("u_drops_beta", "beta * slow[p] +", "slow[p] +", 0),
    ("drops_alpha", "ref - alpha * lr * u", "ref - lr * u", 0),
    ("new_ignores_u", "ref - alpha * lr * u", "avg", 0),
    ("anchor_not_updated", "anchor[p] = fresh;", "", 0),
    ("broadcast_avg", "store_as(param_dt, fresh);", "store_as(param_dt, avg);", 0),
    ("u_not_stored", "slow[p] = u;", "", 0),
    ("replica_index_dropped", "gsum += grads[(int64_t)i * P + p];",
     "gsum += grads[p];", 0),
    ("first_replica_skipped", "for (int i = 0; i < W; ++i) gsum",
     "for (int i = 1; i < W; ++i) gsum", 0),
    ("avg_wrong_divisor", "xsum / (double)W", "xsum / (double)(W + 1)", 0),
    ("avg_of_pre_step_params", "xsum += x;", "xsum += params[k];", 0),
    ("init_mom_not_zero", "mom[(int64_t)i * P + p] = 0.0;",
     "mom[(int64_t)i * P + p] = th;", 0),
    ("init_anchor_zero", "anchor[p] = store_as(aux_dt, th);", "anchor[p] = 0.0;", 0),
    ("bf16_ties_away", "uint32_t lsb = (b >> 16) & 1u;", "uint32_t lsb = 0u;", 0),
    ("f32_rounding_dropped", "return (double)(float)x;", "return x;", 0),
    ("vform_drops_beta", "beta * velocity[p] + delta", "velocity[p] + delta", 0),
    ("vform_delta_sign", "double delta = avg - ref;", "double delta = ref - avg;", 0),
    ("localsgd_not_broadcast", "params[(int64_t)i * P + p] = store_as(param_dt, avg);", ";", 0),
    ("localsgd_anchor_skipped", "if (anchor) anchor[p] = avg;", "", 0),
    ("localsgd_grad_of_replica0", "mu * mom[k] + grads[k]", "mu * mom[k] + grads[p]", 1),
    ("localsgd_avg_wrong_divisor", "store_as(aux_dt, xsum / (double)W)",
     "store_as(aux_dt, xsum / (double)(W + 1))", 0),
    ("ddp_uses_local_grad", "mu * mom[k] + gbar", "mu * mom[k] + grads[k]", 2),
    ("ddp_gbar_not_divided", "gsum / (double)W", "gsum", 2),
    ("ddp_drops_mu", "mu * mom[k] + gbar", "mom[k] + gbar", 2),
    ("sgd_wd_sign", "g + o->wd * *theta", "g - o->wd * *theta", 0),
    ("sgd_wd_dropped", "g + o->wd * *theta", "g", 0),
    ("adamw_decay_dropped", "*theta * decay", "*theta", 0),
    ("adamw_bc1_dropped", "o->lr / bc1", "o->lr", 0),
    ("adamw_bc2_dropped", "sqrt(*v) / sqrt_bc2", "sqrt(*v)", 0),
    ("adamw_m_weight", "(1.0 - o->mu) * g", "g", 0),
    ("adamw_v_not_squared", "(1.0 - o->beta2) * g * g", "(1.0 - o->beta2) * g", 0),
    ("adamw_eps_inside_sqrt", "sqrt(*v) / sqrt_bc2 + o->eps", "sqrt(*v / bc2 + o->eps)", 0),
    ("adamw_step_off_by_one", "pow(o->mu, (double)o->step)", "pow(o->mu, (double)(o->step + 1))", 0),
    ("opt_sync_local_grad", "strategy == 1 ? grads[k] : gbar", "grads[k]", 0),
    ("opt_sync_drops_beta", "beta * slow[p] + (ref - avg) / o->lr", "(ref - avg) / o->lr", 0),
    ("opt_sync_sign", "ref - alpha * o->lr * u", "ref + alpha * o->lr * u", 0),
    ("avg_state_divisor", "msum / (double)W", "msum", 0),
    ("avg_state_skips_mom2", "if (mom2) mom2[(int64_t)i * P + p] = store_as(mom_dt, vsum / (double)W);", "", 0),
    ("write_back_wrong_value", "grads[(int64_t)i * P + p] = gbar;", "grads[(int64_t)i * P + p] = 2.0 * gbar;", 0),
    ("write_back_for_localsgd", "if ((flags & 1u) && strategy != 1)", "if (flags & 1u)", 0),
    # storage-rounding points (Algorithm 1 and Sec. 4.2: a tensor holds its
    # storage type's value from the moment the implementation writes it)
    ("init_theta0_unrounded", "double th = store_as(param_dt, theta0[p]);",
     "double th = theta0[p];", 0),
    ("local_mom_unrounded", "double buf = store_as(mom_dt, mu * mom[k] + grads[k]);",
     "double buf = mu * mom[k] + grads[k];", 0),
    ("local_param_unrounded", "params[k] = store_as(param_dt, params[k] - lr * buf);",
     "params[k] = params[k] - lr * buf;", 0),
    ("reconcile_gbar_unrounded", "double gbar = store_as(aux_dt, gsum / (double)W);",
     "double gbar = gsum / (double)W;", 0),
    ("reconcile_mom_unrounded", "double buf = store_as(mom_dt, mu * mom[k] + gbar);",
     "double buf = mu * mom[k] + gbar;", 0),
    ("reconcile_x_unrounded", "double x = store_as(param_dt, params[k] - lr * buf);",
     "double x = params[k] - lr * buf;", 0),
    ("reconcile_u_unrounded", "double u = store_as(aux_dt, beta * slow[p] + (ref - avg) / lr);",
     "double u = beta * slow[p] + (ref - avg) / lr;", 0),
    ("reconcile_new_unrounded", "double fresh = store_as(aux_dt, ref - alpha * lr * u);",
     "double fresh = ref - alpha * lr * u;", 0),
    ("reconcile_broadcast_unrounded", "params[(int64_t)i * P + p] = store_as(param_dt, fresh);",
     "params[(int64_t)i * P + p] = fresh;", 0),
    ("vform_gbar_unrounded", "double gbar = store_as(aux_dt, gsum / (double)W);",
     "double gbar = gsum / (double)W;", 1),
    ("vform_mom_unrounded", "double buf = store_as(mom_dt, mu * mom[k] + gbar);",
     "double buf = mu * mom[k] + gbar;", 1),
    ("vform_x_unrounded", "xsum += store_as(param_dt, params[k] - lr * buf);",
     "xsum += params[k] - lr * buf;", 0),
    ("vform_v_unrounded", "double v = store_as(aux_dt, beta * velocity[p] + delta);",
     "double v = beta * velocity[p] + delta;", 0),
    ("vform_new_unrounded", "double fresh = store_as(aux_dt, ref + v);",
     "double fresh = ref + v;", 0),
    ("vform_broadcast_unrounded", "params[(int64_t)i * P + p] = store_as(param_dt, fresh);",
     "params[(int64_t)i * P + p] = fresh;", 1),
    ("localsgd_mom_unrounded", "double buf = store_as(mom_dt, mu * mom[k] + grads[k]);",
     "double buf = mu * mom[k] + grads[k];", 1),
    ("localsgd_x_unrounded", "xsum += store_as(param_dt, params[k] - lr * buf);",
     "xsum += params[k] - lr * buf;", 1),
    ("localsgd_avg_unrounded", "double avg = store_as(aux_dt, xsum / (double)W);",
     "double avg = xsum / (double)W;", 0),
    ("localsgd_broadcast_unrounded", "params[(int64_t)i * P + p] = store_as(param_dt, avg);",
     "params[(int64_t)i * P + p] = avg;", 0),
    ("ddp_gbar_unrounded", "double gbar = store_as(aux_dt, gsum / (double)W);",
     "double gbar = gsum / (double)W;", 2),
    ("ddp_mom_unrounded", "double buf = store_as(mom_dt, mu * mom[k] + gbar);",
     "double buf = mu * mom[k] + gbar;", 2),
    ("ddp_param_unrounded", "params[k] = store_as(param_dt, params[k] - lr * buf);",
     "params[k] = params[k] - lr * buf;", 1),
    ("opt_gbar_unrounded", "\n            gbar = store_as(aux_dt, gsum / (double)W);",
     "\n            gbar = gsum / (double)W;", 0),
    ("opt_sgd_decayed_grad_unrounded", "store_as(grad_dt, g + o->wd * *theta)",
     "(g + o->wd * *theta)", 0),
    ("opt_sgd_mom_unrounded", "*m = store_as(mom_dt, o->mu * *m + d);", "*m = o->mu * *m + d;", 0),
    ("opt_sgd_param_unrounded", "*theta = store_as(param_dt, *theta - o->lr * *m);",
     "*theta = *theta - o->lr * *m;", 0),
    ("opt_u_unrounded", "double u = store_as(aux_dt, beta * slow[p] + (ref - avg) / o->lr);",
     "double u = beta * slow[p] + (ref - avg) / o->lr;", 0),
    ("opt_new_unrounded", "fresh = store_as(aux_dt, ref - alpha * o->lr * u);",
     "fresh = ref - alpha * o->lr * u;", 0),
    ("opt_broadcast_unrounded", "params[(int64_t)i * P + p] = store_as(param_dt, fresh);",
     "params[(int64_t)i * P + p] = fresh;", 2),
    ("opt_localsgd_avg_unrounded", "fresh = store_as(aux_dt, avg);", "fresh = avg;", 0),
    ("opt_avg_state_unrounded", "mom[(int64_t)i * P + p] = store_as(mom_dt, msum / (double)W);",
     "mom[(int64_t)i * P + p] = msum / (double)W;", 0),
    ("opt_avg_state_mom2_unrounded", "mom2[(int64_t)i * P + p] = store_as(mom_dt, vsum / (double)W);",
     "mom2[(int64_t)i * P + p] = vsum / (double)W;", 0),
    ("adamw_decay_factor_exact", "double decay = store_as(grad_dt, 1.0 - o->lr * o->wd);",
     "double decay = 1.0 - o->lr * o->wd;", 0),
    ("adamw_decayed_param_unrounded", "store_as(param_dt, *theta * decay)", "(*theta * decay)", 0),
    ("adamw_m_unrounded", "*m = store_as(mom_dt, o->mu * *m + (1.0 - o->mu) * g);",
     "*m = o->mu * *m + (1.0 - o->mu) * g;", 0),
    ("adamw_v_unrounded", "*v = store_as(mom_dt, o->beta2 * *v + (1.0 - o->beta2) * g * g);",
     "*v = o->beta2 * *v + (1.0 - o->beta2) * g * g;", 0),
    ("adamw_step_size_exact", "double step_size = store_as(grad_dt, o->lr / bc1);",
     "double step_size = o->lr / bc1;", 0),
    ("adamw_sqrt_bc2_exact", "double sqrt_bc2 = store_as(grad_dt, sqrt(bc2));",
     "double sqrt_bc2 = sqrt(bc2);", 0),
    ("adamw_param_unrounded", "*theta = store_as(param_dt, th - step_size * *m / denom);",
     "*theta = th - step_size * *m / denom;", 0),
]

# mutants that edit several places at once: (name, [(old, new, occurrence), ...])
MULTI_MUTANTS = [
    ("adamw_scalars_exact",
     [("double decay = store_as(grad_dt, 1.0 - o->lr * o->wd);", "double decay = 1.0 - o->lr * o->wd;", 0),
      ("double step_size = store_as(grad_dt, o->lr / bc1);", "double step_size = o->lr / bc1;", 0),
      ("double sqrt_bc2 = store_as(grad_dt, sqrt(bc2));", "double sqrt_bc2 = sqrt(bc2);", 0)]),
    ("rounding_dropped_everywhere",
     [("if (dt == ORACLE_F32) return round_to_f32(x);", "if (dt == ORACLE_F32) return x;", 0),
      ("if (dt == ORACLE_BF16) return round_to_bf16(x);", "if (dt == ORACLE_BF16) return x;", 0)]),
]


def _mutate(src, old, new, occ):
    parts = src.split(old)
    assert len(parts) > occ + 1, f"mutation site {old!r} not found"
    return old.join(parts[: occ + 1]) + new + old.join(parts[occ + 1:])


INDEPENDENT_PINS = [p for p in oracle_pins.ALL_PINS
                    if p is not oracle_pins.pin_general_sgd_matches_plain]

ALL_MUTANTS = [(name, [(old, new, occ)]) for name, old, new, occ in MUTANTS] + MULTI_MUTANTS


def test_mutant_names_are_unique():
    names = [m[0] for m in ALL_MUTANTS]
    assert len(names) == len(set(names))


@pytest.mark.parametrize("name,edits", ALL_MUTANTS, ids=[m[0] for m in ALL_MUTANTS])
def test_mutant_is_caught(tmp_path, name, edits):
    src = open(SRC).read()
    mutated = src
    for old, new, occ in edits:
        mutated = _mutate(mutated, old, new, occ)
    assert mutated != src
    c_path = tmp_path / f"{name}.c"
    c_path.write_text(mutated)
    lib = oracle.load(oracle.build(str(c_path), str(tmp_path / f"lib{name}.so")))
    caught = []
    for pin in INDEPENDENT_PINS:
        try:
            pin(use=lib)
        except (AssertionError, ValueError, FloatingPointError) as e:
            caught.append((pin.__name__, str(e)[:80]))
            break
    assert caught, f"mutant {name} passed every independent pin"
