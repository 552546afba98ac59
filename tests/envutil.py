"""Create an ensemble handle with some RAFIKI_* switches set for create only (they are
read by rafiki_ensemble_create; the environment is restored afterwards)."""
import os

from paper_1804_06087_amd import Ensemble

# the layer-by-layer path with every model on its own stream: no whole-network kernel,
# no grouped launches (the schedules, tile forcing and grouping tests need it)
LAYER_PATH = {"RAFIKI_FUSED_NET": "0", "RAFIKI_GROUPED": "0"}


def create(env, specs, params, precision="bf16", max_batch=64):
    old = {k: os.environ.get(k) for k in env}
    os.environ.update(env)
    try:
        return Ensemble(specs, params, precision=precision, max_batch=max_batch)
    finally:
        for k, v in old.items():
            if v is None:
                del os.environ[k]
            else:
                os.environ[k] = v
