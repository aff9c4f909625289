"""MI355X-native replica-batched simulation of a learned prefill/decode router.

Importing the package is cheap: the HIP library binding lives in
``paper_2609_16206_amd.rt_router`` and is loaded only when that module is
imported.
"""
__all__ = ["workload"]
