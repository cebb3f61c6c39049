"""MI355X-native VLA serving hot path: VLM prefill producing a per-layer prefix
KV cache, the action diffusion transformer's Euler loop, stage co-execution on
CU-masked HIP streams, and an SLO-aware host scheduler.

The compute lives in ``libvla.so`` (HIP kernels for gfx950 behind a C ABI);
``paper_2609_12075_amd.vla`` is the thin ctypes binding. Importing the package
loads nothing; the binding loads the library on first use and raises if it
has not been built.
"""
__all__ = ["synth", "vla"]
