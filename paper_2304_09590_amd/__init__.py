"""MI355X-native parallel neural network (PNN) training path: K child networks trained by
back-propagation and SGD on their own slices of the data, merged by averaging (Kalwarowskyj &
Schikuta, "Parallel Neural Networks in Golang").  The compute runs in the HIP library
libpnn.so; this package holds its sources (csrc/), the build step and the ctypes binding."""
from .pnn import PNN, PnnConfig, PnnError, config_from_workload, make_config, param_count, shard  # noqa: F401
