"""Seeded synthetic inputs shared by the HIP path's tests and benchmark and by
the CPU oracle's tests.  Draws numbers and describes workload shapes only; it
holds none of the method's arithmetic."""
