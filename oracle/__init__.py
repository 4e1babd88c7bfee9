"""CPU float64 oracle of the parallel-window neural decoder.

Test infrastructure only: the test-suite, the smoke check and the CPU baseline leg of the
benchmark may import it; the HIP product path never does and shares no code with it.
"""
