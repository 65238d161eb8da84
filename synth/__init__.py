"""Seeded synthetic inputs shared by the tests, the oracle checks and the benchmark.

Holds no attention arithmetic: only random draws, dtype rounding, the fp8 key
quantisation that produces the cache contents, and cache layouts."""
from .gen import normal, normal_at, permutation, splitmix64, stream_key, uniform_int  # noqa: F401
from .workloads import (FULLKEY, INT4KEY, WORKLOADS, DecodeSpec, PrefillSpec, make_decode,  # noqa: F401
                        make_prefill, make_prefill_grad, quantize_e4m3, quantize_int4, with_shape)
