"""Oracle (test infrastructure only): a plain fp64 CPU statement of the probe forward."""
