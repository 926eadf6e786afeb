"""MI355X (gfx950) rollout hot path of FinRL-Podracer (arXiv 2111.05188).

``tp``      : Python binding of the C ABI in include/tp.h (libtp.so).
``problem`` : device-side setup of a workload (market, state, actor, store).
``build``   : compiles libtp.so for gfx950.
"""
