"""Plain, slow, fp64 CPU oracle of the ensemble-inference hot path and of the greedy
batch-size scheduler around it.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's CPU
baseline may import this package; the product path never calls it and shares no
code with it.
"""
from .reference import (to_bf16_rne, conv2d, batchnorm, relu, maxpool2d, global_avgpool, fc,
                        embedding, conv1d_maxtime, concat, softmax, combine_mean, argmax_first,
                        run_model, ensemble, model_macs, combine_vote, ensemble_vote)
from .scheduler import greedy_decide, simulate_greedy, simulate_greedy_multi, serving_stats
from . import rl

__all__ = ["to_bf16_rne", "conv2d", "batchnorm", "relu", "maxpool2d", "global_avgpool", "fc",
           "embedding", "conv1d_maxtime", "concat", "softmax", "combine_mean", "argmax_first",
           "run_model", "ensemble", "model_macs", "combine_vote", "ensemble_vote",
           "greedy_decide", "simulate_greedy", "simulate_greedy_multi", "serving_stats", "rl"]
