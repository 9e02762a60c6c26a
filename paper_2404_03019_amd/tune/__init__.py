"""Offline tuning of the kernel selector: sweep (GPU) -> performance database -> decision trees -> C++ if/else."""
