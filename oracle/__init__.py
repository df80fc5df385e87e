"""CPU oracle for the quantized LSTM path -- test infrastructure only.

Imported by tests/, the smoke check and the benchmark's CPU-baseline leg; the
GPU library never imports or links it.
"""
