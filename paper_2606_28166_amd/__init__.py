"""MI355X-native tandem co-generation rollout (Tandem RL with Verifiable Rewards).

libtandem.so (hand-written HIP for gfx950 behind the C ABI of include/tandem.h)
runs the hot path: the dual-model decode step with owner sampling, senior
log-probs and the handoff rule, plus the prefill of both models.  Python only
marshals arguments and lets PyTorch allocate device memory:

    from paper_2606_28166_amd import engine      # loads libtandem.so (raises if unbuilt)
"""
__all__ = ["engine"]
