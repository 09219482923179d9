"""ROCKET oracle package -- test infrastructure only (see rocket_oracle.py)."""
