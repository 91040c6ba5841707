"""Seeded synthetic inputs (profiles, sequence databases) for the search."""
from .gen import *  # noqa: F401,F403
from .gen import (ALPHABET, BACKGROUND, Database, Profile, Workload, WORKLOADS,
                  make_profile, make_database, random_sequences, sample_homologs,
                  workload_profile, workload_database, c4_profiles)
