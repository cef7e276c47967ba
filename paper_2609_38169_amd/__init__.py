"""MI355X-native fused decode step over a pool of quantized gated-Delta
recurrent states (STEPQuant's data-parallel hot path).

    from paper_2609_38169_amd import stepq      # ctypes binding of libstepq
    from paper_2609_38169_amd import workloads  # seeded synthetic inputs
"""
