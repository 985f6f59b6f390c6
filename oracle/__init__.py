"""CPU oracle of the scheduling-decision path: test infrastructure only.

Only tests, the smoke check and the benchmark's CPU-baseline leg may use it;
the HIP path never imports it and it imports nothing from the product package.
"""
from .sage_oracle import (attained_service, bf16_to_f64, bin_of, cost, cost_variant,  # noqa: F401
                          gittins, gittins_attained, histogram, length_similarity, mean_index, mix_uniform,
                          predict, predict_by_length, rank, round_to_bf16, schedule, search, similarity, store_insert, topk,
                          topk_row)
from .sage_sim import (POLICIES, policy_order, refresh_levels, service_cost, simulate,  # noqa: F401
                       simulate_policy)
