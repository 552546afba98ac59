"""MI355X (gfx950) ensemble-inference hot path: HIP kernels behind a C ABI
(``include/rafiki_ensemble.h``), the greedy batch-size scheduler and serving loops
(``include/rafiki_sched.h``), the actor-critic scheduler (``include/rafiki_rl.h``), and a
thin ctypes binding."""
from .binding import (Ensemble, RafikiError, load_library, last_error, LIB_PATH, EXPORTED,
                      RAFIKI_OK, RAFIKI_ERR_INVALID, RAFIKI_ERR_UNSUPPORTED, RAFIKI_ERR_NOMEM,
                      RAFIKI_ERR_HIP, RAFIKI_FP32, RAFIKI_BF16, RAFIKI_TILE_DIRECT, greedy_decide, greedy_simulate,
                      greedy_simulate_multi, RLScheduler)

__all__ = ["Ensemble", "RafikiError", "load_library", "last_error", "LIB_PATH", "EXPORTED", "RAFIKI_OK",
           "RAFIKI_ERR_INVALID", "RAFIKI_ERR_UNSUPPORTED", "RAFIKI_ERR_NOMEM", "RAFIKI_ERR_HIP",
           "RAFIKI_FP32", "RAFIKI_BF16", "RAFIKI_TILE_DIRECT", "greedy_decide", "greedy_simulate",
           "greedy_simulate_multi", "RLScheduler"]
