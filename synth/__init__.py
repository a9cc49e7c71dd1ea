"""Seeded synthetic inputs for the GBA push-step: counter-based values, Zipf
IDs, staleness draws and the five workload shapes.  Holds none of the
aggregation arithmetic; both the oracle's tests and the device path draw their
inputs here."""
from . import configs, counter, workload, zipf  # noqa: F401
