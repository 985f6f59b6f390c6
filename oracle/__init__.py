"""CPU oracle of the scheduling-decision path: test infrastructure only.

Only tests, the smoke check and the benchmark's CPU-baseline leg may use it;
the HIP path never imports it and it imports nothing from the product package.
"""
from .sage_oracle import (attained_service, bf16_to_f64, bin_of, cost, gittins,  # noqa: F401
                          gittins_attained, histogram, predict, rank, round_to_bf16, schedule,
                          search, similarity, topk, topk_row)
