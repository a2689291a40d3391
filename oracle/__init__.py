"""CPU oracle of the TurboESM KV-cache path. Test infrastructure only: used by
tests/, __graft_entry__.smoke() and the CPU-baseline leg of bench.py."""
